#!/usr/bin/env python3
"""Benchmark of the resistance-curvature hot path on one MI355X.

One step = the whole path over one synthetic graph: resistance for all K projection
columns (right-hand sides, batched CG, edge-distance accumulation), node and edge
curvature, and the node/edge sampling probabilities.  Inputs are resident in HBM
before the timed region starts.  Prints ONE JSON line on stdout; progress goes to
stderr.

    python bench.py [--steps K] [--warmup W] [--config cl2400k] [--no-cpu-baseline]

After the timed steps it also times one curvature-guided training subgraph per
distribution (erc_draw + erc_subgraph; not part of a step) unless --no-draw.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0  # MI355X HBM3E, published

# L2-to-fabric traffic of one full SpMM launch on the 2.4M-node workload, from two
# rocprofv3 --pmc runs of this benchmark (FETCH_SIZE, then WRITE_SIZE, KiB per
# dispatch, median over full launches), each scaled by what the counter reads for a
# plain copy kernel of known size run in the same process (FETCH_SIZE x 2.0,
# WRITE_SIZE x 1.0).  The counters count every request that leaves the L2, served by
# the Infinity Cache or by HBM alike.  Valid only for the sources it was measured on:
# reported as null once they change (the hash is only ever updated with new counters).
MEASURED_TRAFFIC = {
    "workload": "cl2400k",
    "source_sha256_16": "bead0a370a8ed9f7",
    "fetch_bytes": 32563989888,
    "write_bytes": 664731648,
    "profile": "profiles/k_spmm_cl2400k.md",
}


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def elem_bytes(dtype: str) -> int:
    return 4 if dtype == "f32" else 8


def spmm_bytes_per_launch(g, kb: int, dtype: str) -> int:
    """Compulsory bytes of one SpMM launch: column indices (4 B per stored entry) and,
    on weighted graphs, weights in the working precision, row pointers, one n-vector of
    the diagonal, one read of p and one write of q (n x kb each).  Neighbour-row gathers
    beyond that one read of p are not counted."""
    s = elem_bytes(dtype)
    per_nnz = 4 + (s if g.w is not None else 0)
    return per_nnz * g.nnz + 8 * (g.n + 1) + s * g.n + 2 * s * g.n * kb


def spmm_fused_bytes_per_launch(g, kb: int, dtype: str) -> int:
    """What this SpMM kernel reads and writes once: column indices (+ weights), row
    pointers, p, r (read for the fused r.q) and q; it forms q_i = delta p_i +
    sum_j w_ij (p_i - p_j) without a stored diagonal."""
    s = elem_bytes(dtype)
    per_nnz = 4 + (s if g.w is not None else 0)
    return per_nnz * g.nnz + 8 * (g.n + 1) + 3 * s * g.n * kb


def iteration_bytes(g, kb: int, dtype: str) -> int:
    """Algorithmic bytes of one CG iteration of one block: 4 nnz (+ s nnz) + 8 (n+1) +
    s n + 11 s n kb, i.e. the SpMM's compulsory bytes and the vector passes of a
    textbook iteration (SpMM: p read, q written; z, r update: z, p, r, q read, z, r
    written; p update: r, p read, p written).  The fused kernels here make 10 passes."""
    s = elem_bytes(dtype)
    per_nnz = 4 + (s if g.w is not None else 0)
    return per_nnz * g.nnz + 8 * (g.n + 1) + s * g.n + 11 * s * g.n * kb


def kernel_source_hash() -> str:
    """sha256 (first 16 hex digits) of the SpMM's kernel source and of the host code
    that plans its launch; stored counter values are used only while both match."""
    import hashlib

    h = hashlib.sha256()
    for name in ("erc_kernels.hip", "erc_host.cpp"):
        with open(os.path.join(ROOT, "paper_2609_27209_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def padded(kb: int, dtype: str) -> int:
    w = 16 if dtype == "f32" else 8
    while w < kb:
        w *= 2
    return w


_CPU = {}


def _cpu_init():
    from threadpoolctl import threadpool_limits

    threadpool_limits(limits=1)  # one thread per oracle process


def _cpu_rhs(args):
    from oracle import erc as OE

    c0, nc = args
    gs, p = _CPU["g"], _CPU["p"]
    return c0, OE.rhs(gs, p.K, c0, nc, p.seed, p.dtype)


def _cpu_cg(args):
    from oracle import erc as OE

    c0, c1 = args
    res = OE.cg_columns(_CPU["L"], _CPU["p"].delta, _CPU["Y"][:, c0:c1], 1e-300, _CPU["iters"])
    return c0, res.Z


def host_cpu():
    """CPU model, logical CPUs and the CPUs this process may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count() or 1
    return {"model": model, "nproc": os.cpu_count() or 1, "usable": usable}


def cpu_baseline(g, p, wl, iters_total: int, scale_div: int = 25, cg_iters: int = 16,
                 procs: int = 0):
    """Time the CPU oracle, column-parallel on the host's cores, on a bounded sample of
    this workload and scale to edges/s.

    Sample: a 1/`scale_div` instance of the same graph recipe (n and m divided by
    `scale_div`, the generator's offset i0 scaled with n).  The oracle runs one block of
    right-hand sides and `cg_iters` CG iterations of one full block split into column
    ranges over `procs` processes (one thread each; the columns are independent, as in
    Algorithm 1), and Laplacian assembly, one block of edge distances, curvature and
    sampling in one process.  Each stage is scaled linearly in the graph size (stored
    entries or edges), RHS and distances by the number of blocks, and CG by the
    column-iterations the GPU run took.
    """
    import multiprocessing as mp

    import numpy as np

    import gen
    from oracle import erc as OE
    from oracle import graph as OG

    cpu = host_cpu()
    procs = procs or min(16, cpu["usable"])
    kb = p.k_block
    nblocks = math.ceil(p.K / kb)
    args = dict(wl.graph_args)
    if wl.graph_kind == "chung_lu":
        args.update(n=max(1000, args["n"] // scale_div), m_target=max(2000, args["m_target"] // scale_div),
                    i0=args["i0"] / scale_div)
        gs = gen.graphs.chung_lu(**args)
    else:
        gs = g
    f_m = g.m / gs.m
    f_nnz = g.nnz / gs.nnz
    t_wall0 = time.perf_counter()
    t0 = time.perf_counter()
    L = OG.laplacian(gs)
    eu, ev, _ = OG.canonical_edges(gs)
    t_setup = (time.perf_counter() - t0) * f_m
    _CPU.update(g=gs, p=p, L=L, iters=cg_iters)
    bounds = [(kb * k) // procs for k in range(procs + 1)]
    ranges = [(bounds[k], bounds[k + 1]) for k in range(procs) if bounds[k + 1] > bounds[k]]
    ctx = mp.get_context("fork")
    with ctx.Pool(len(ranges), initializer=_cpu_init) as pool:
        t0 = time.perf_counter()
        parts = sorted(pool.map(_cpu_rhs, [(a, b - a) for a, b in ranges]))
        t_rhs_s = time.perf_counter() - t0
        Y = np.concatenate([y for _, y in parts], axis=1)
        _CPU["Y"] = Y
    # a fresh pool so the workers see Y (fork after it is set)
    with ctx.Pool(len(ranges), initializer=_cpu_init) as pool:
        t0 = time.perf_counter()
        zs = sorted(pool.map(_cpu_cg, ranges))
        t_cg_s = time.perf_counter() - t0
    Z = np.concatenate([z for _, z in zs], axis=1)
    t_rhs = t_rhs_s * f_nnz * nblocks
    t_it = t_cg_s / cg_iters * f_nnz
    t_cg = t_it * iters_total / kb
    from threadpoolctl import threadpool_limits

    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        R = OE.edge_distances(Z, eu, ev)
        t_dist = (time.perf_counter() - t0) * f_m * nblocks
        t0 = time.perf_counter()
        _, kappa = OE.curvature(gs, R)
        OE.sampling_probs(gs, kappa, p.eta)
        t_curv = (time.perf_counter() - t0) * f_m
    wall = time.perf_counter() - t_wall0
    _CPU.clear()
    total = t_setup + t_rhs + t_cg + t_dist + t_curv
    log(f"cpu baseline: estimated {total:.0f}s for the full workload on {len(ranges)} processes")
    sample = (f"oracle (fp64 NumPy/SciPy) on a 1/{scale_div} instance of the same recipe "
              f"({gs.n} nodes, {gs.m} edges): RHS of one {kb}-column block and {cg_iters} CG "
              f"iterations of it in {len(ranges)} column ranges on {len(ranges)} processes "
              f"({t_rhs_s:.1f}s, {t_cg_s:.1f}s measured), Laplacian assembly, edge distances, "
              f"curvature and sampling on one; scaled by edges or stored entries: assembly "
              f"{t_setup:.1f}s, RHS x {nblocks} blocks {t_rhs:.1f}s, CG {t_it:.2f}s per "
              f"block-iteration x {iters_total} column-iterations / {kb} = {t_cg:.0f}s, edge "
              f"distances {t_dist:.1f}s, curvature + sampling {t_curv:.1f}s; estimated full "
              f"run {total:.0f}s")
    return {"value": g.m / total, "unit": "edges/s", "cores": len(ranges), "kind": "oracle",
            "sample": sample, "est_seconds": round(total, 1),
            "sample_measured_s": round(wall, 1), "cpu_model": cpu["model"],
            "nproc": cpu["nproc"], "usable_cpus": cpu["usable"],
            "processes": len(ranges)}


def gather_ceiling(g, kb: int, dtype: str, torch, reps: int = 5, streams=None):
    """Time the gather probe (erc_probe_gather) replaying index streams over a table of
    the p block's size (n rows of kb working-precision values): the SpMM's own column
    indices by default, or the named streams of `streams` (name -> int32 array,
    footprint in rows).  Median of `reps` launches after one warm-up, HIP events on the
    stream the probe runs on."""
    import numpy as np

    from paper_2609_27209_amd import _abi

    row_bytes = kb * elem_bytes(dtype)
    if streams is None:
        streams = {"spmm_column_indices": (np.asarray(g.col, np.int32), g.n)}
    rows_max = max(r for _, r in streams.values())
    table = torch.empty(rows_max * row_bytes // 4, dtype=torch.float32, device="cuda")
    table.uniform_()
    out = {}
    st = torch.cuda.current_stream()
    for name, (idx_np, rows) in streams.items():
        idx = torch.from_numpy(np.ascontiguousarray(idx_np, np.int32)).cuda()
        res = torch.empty(_abi.erc_probe_out_bytes(idx.numel(), row_bytes) // 4,
                          dtype=torch.float32, device="cuda")
        ts = []
        for r in range(reps + 1):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(st)
            _abi.erc_probe_gather(idx.data_ptr(), idx.numel(), table.data_ptr(), rows, row_bytes,
                                  res.data_ptr(), st.cuda_stream)
            e1.record(st)
            torch.cuda.synchronize()
            if r > 0:
                ts.append(e0.elapsed_time(e1))
        ms = sorted(ts)[len(ts) // 2]
        gathered = idx.numel() * row_bytes
        out[name] = {"ms": round(ms, 4), "gathered_bytes": gathered,
                     "gbs": round(gathered / (ms / 1e3) / 1e9, 1),
                     "footprint_bytes": rows * row_bytes}
        log(f"gather probe {name}: {out[name]}")
        del idx, res
    del table
    return out


def relabelled_step(g, p, torch, seed: int = 7):
    """One step (resistance + curvature + sampling probabilities) on a copy of the
    graph with node ids randomly permuted: the same degree sequence and structure in an
    order with no hub-first locality.  Times the step and its SpMM launches."""
    import numpy as np

    import gen
    import paper_2609_27209_amd as E

    t0 = time.perf_counter()
    gr = gen.relabel(g, np.random.default_rng(seed).permutation(g.n))
    t_relabel = time.perf_counter() - t0
    G = E.Graph(gr.rowptr, gr.col, gr.w, solve_dtype=p.dtype)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    R, info = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed, profile=True)
    _, kk = G.curvature(R)
    G.sampling_probs(kk, p.eta)
    torch.cuda.synchronize()
    sec = time.perf_counter() - t0
    avg = info["ms_spmm"] / max(info["spmm_full"], 1)
    G.close()
    del G, R, kk
    out = {"permutation_seed": seed, "ms_per_step": round(sec * 1e3, 1),
           "edges_per_s": g.m / sec, "iters_max": info["iters_max"],
           "spmm_avg_ms": round(avg, 4), "relabel_host_s": round(t_relabel, 1)}
    log(f"relabelled copy: {out}")
    return out


def subgraph_draw(G, pn, pe, torch, reps: int = 5):
    """Time one curvature-guided training subgraph per distribution, outside the timed
    steps: erc_draw (1% of the nodes, or 0.1% of the edges, as draws) then erc_subgraph
    on the probabilities of the last step, median over `reps` with HIP events."""
    out = {}
    for items, prob, draws in (("nodes", pn, max(1, G.n // 100)),
                               ("edges", pe, max(1, G.m // 1000))):
        ts, sizes = [], None
        for r in range(reps + 1):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            idx = G.draw(items, prob, draws, seed=1000 + r)
            sg = G.subgraph(items, idx)
            e1.record()
            torch.cuda.synchronize()
            if r > 0:
                ts.append(e0.elapsed_time(e1))
            sizes = (sg["nodes"].numel(), sg["edges"].numel())
        ts.sort()
        out[items] = {"draws": draws, "ms": round(ts[len(ts) // 2], 3),
                      "subgraph_nodes": sizes[0], "subgraph_edges": sizes[1]}
        log(f"subgraph draw ({items}): {out[items]}")
    return out


def jacobi_variant(G, g, p, R_plain, torch):
    """One step of the same path with the Jacobi-preconditioned CG variant (ERC_JACOBI;
    not the paper's method, not part of `value`): edges/s, iterations, and how far its
    R lies from the plain-CG R of the last timed step (both stop at the same residual
    tolerance, so the difference is the two solves' truncation errors)."""
    import time as _t

    torch.cuda.synchronize()
    t0 = _t.perf_counter()
    R, info = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed,
                           precond="jacobi")
    _, kk = G.curvature(R)
    G.sampling_probs(kk, p.eta)
    torch.cuda.synchronize()
    sec = _t.perf_counter() - t0
    rel = ((R - R_plain).abs() / R_plain)[::7].float()
    q = torch.quantile(rel[: 1 << 24], torch.tensor([0.5, 0.999], device=rel.device))
    out = {"value": g.m / sec, "unit": "edges/s", "ms_per_step": round(sec * 1e3, 1),
           "iters_max": info["iters_max"], "iters_total": info["iters_total"],
           "max_final_relres": info["max_final_relres"],
           "R_rel_diff_vs_plain": {"median": float(q[0]), "p99.9": float(q[1]),
                                   "max": float(((R - R_plain).abs() / R_plain).max())}}
    log(f"jacobi variant: {out}")
    return out


def per_config_table(steps: int, warmup: int, only=None):
    """Every workload at its own solve parameters: curvature edges/s and m*K/s end to
    end (resistance + curvature + sampling probabilities, inputs in HBM), with and
    without HIP-graph replay of the iteration groups, iterations,
    average SpMM launch, one step of the Jacobi variant (time and iterations; one run,
    after the timed steps), and the device memory the caller allocates (graph buffer,
    workspace, R, p, kappa and both probability vectors, sampling scratch) for block
    widths 32..256 (the paper's Table 3 reports peak memory against its batch size b)."""
    import torch

    import gen
    import paper_2609_27209_amd as E
    from paper_2609_27209_amd import _abi

    rows = []
    for name in gen.configs.ORDER:
        if only and name not in only:
            continue
        wl = gen.CONFIGS[name]
        p = wl.params
        g = gen.make_graph(name, progress=log)
        G = E.Graph(g.rowptr, g.col, g.w, solve_dtype=p.dtype)

        def step(profile, graph=True):
            R, info = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed,
                                   profile=profile, graph=graph)
            _, kk = G.curvature(R)
            G.sampling_probs(kk, p.eta)
            return info

        for _ in range(warmup):
            step(False)
        # timed steps as a caller runs them (iteration groups replayed as HIP graphs),
        # the same steps with every launch enqueued separately, then one step with the
        # SpMM launches timed by events (which enqueues them separately too)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            step(False)
        torch.cuda.synchronize()
        sec = (time.perf_counter() - t0) / steps
        t0 = time.perf_counter()
        for _ in range(steps):
            step(False, graph=False)
        torch.cuda.synchronize()
        sec_nograph = (time.perf_counter() - t0) / steps
        infos = [step(True)]
        full = sum(i["spmm_full"] for i in infos)
        avg = sum(i["ms_spmm"] for i in infos) / max(full, 1)
        kb = padded(p.k_block, p.dtype)
        bl = spmm_bytes_per_launch(g, kb, p.dtype)
        # R, kappa and edge probabilities (m fp64 each); p and node probabilities (n each)
        outputs = 8 * (3 * g.m + 2 * g.n) + _abi.erc_sampling_scratch_bytes(G.handle)
        widths = [b for b in (32, 64, 128, 256) if p.dtype == "f32" or b <= 128]
        torch.cuda.synchronize()
        tj = time.perf_counter()
        Rj, ij = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed,
                              precond="jacobi")
        _, kj = G.curvature(Rj)
        G.sampling_probs(kj, p.eta)
        torch.cuda.synchronize()
        sec_j = time.perf_counter() - tj
        del Rj, kj
        desc, keep = E._desc(g.rowptr, g.col, g.w, p.dtype)
        gbytes = _abi.erc_graph_bytes(desc)
        del desc, keep
        mem = {str(b): gbytes + _abi.erc_workspace_bytes(G.handle, b) + outputs for b in widths}
        rows.append({"workload": name, "n": g.n, "m": g.m, "K": p.K, "k_block": p.k_block,
                     "dtype": p.dtype, "ms_per_step": round(sec * 1e3, 2),
                     "ms_per_step_without_graphs": round(sec_nograph * 1e3, 2),
                     "edges_per_s": g.m / sec, "edge_columns_per_s": g.m * p.K / sec,
                     "iters_max": infos[-1]["iters_max"],
                     "spmm_avg_ms": round(avg, 4),
                     "spmm_algorithmic_gbs": round(bl / (avg / 1e3) / 1e9, 1) if full else None,
                     "device_bytes_by_block_width": mem,
                     "jacobi": {"ms_per_step": round(sec_j * 1e3, 2),
                                "iters_max": ij["iters_max"]}})
        log(f"{name}: {rows[-1]}")
        G.close()
        del G, g
    return {"table": "per_config", "steps": steps, "warmup": warmup, "rows": rows}


def block_sweep(name: str, widths):
    """The paper's Table 3 experiment on one workload: the same resistance + curvature +
    sampling-probability step at several block widths b (columns per CG block; K, the
    shift, the tolerance and the seed unchanged), one step each after one warm-up block:
    ms per step, iterations, average SpMM launch and its algorithmic rate, and the
    device memory the caller allocates at that b (graph buffer, workspace, outputs,
    sampling scratch)."""
    import torch

    import gen
    import paper_2609_27209_amd as E
    from paper_2609_27209_amd import _abi

    wl = gen.CONFIGS[name]
    p = wl.params
    g = gen.make_graph(name, progress=log)
    G = E.Graph(g.rowptr, g.col, g.w, solve_dtype=p.dtype)
    desc, keep = E._desc(g.rowptr, g.col, g.w, p.dtype)
    gbytes = _abi.erc_graph_bytes(desc)
    del desc, keep
    outputs = 8 * (3 * g.m + 2 * g.n) + _abi.erc_sampling_scratch_bytes(G.handle)
    G.resistance(p.K, widths[0], p.delta, p.tol, p.max_iter, p.seed, col_begin=0,
                 col_end=widths[0])
    rows = []
    for b in widths:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        R, info = G.resistance(p.K, b, p.delta, p.tol, p.max_iter, p.seed, profile=True)
        _, kk = G.curvature(R)
        G.sampling_probs(kk, p.eta)
        torch.cuda.synchronize()
        sec = time.perf_counter() - t0
        avg = info["ms_spmm"] / max(info["spmm_full"], 1)
        bl = spmm_bytes_per_launch(g, padded(b, p.dtype), p.dtype)
        rows.append({"k_block": b, "blocks": info["blocks"], "ms_per_step": round(sec * 1e3, 1),
                     "edges_per_s": g.m / sec, "iters_max": info["iters_max"],
                     "iters_total": info["iters_total"], "spmm_launches": info["spmm_full"],
                     "spmm_avg_ms": round(avg, 4),
                     "spmm_algorithmic_gbs": round(bl / (avg / 1e3) / 1e9, 1),
                     "device_bytes": gbytes + _abi.erc_workspace_bytes(G.handle, b) + outputs})
        log(f"{name} b={b}: {rows[-1]}")
        del R, kk
    G.close()
    return {"table": "block_sweep", "workload": name, "n": g.n, "m": g.m, "K": p.K,
            "dtype": p.dtype, "rows": rows}


def gather_footprints(name: str, torch):
    """The gather probe's rate for 256-byte-class rows (the workload's p block) on: the
    SpMM's own column indices; the same indices folded into a footprint of F rows (j mod
    F), which fits one XCD's L2, all L2s, or the Infinity Cache; the same indices in a
    random order (no row-order locality); sorted (each row's gathers adjacent: the
    compulsory bytes from the cache); the hub rows (ids below 131072) and the rest
    separately; and uniform indices over footprints beyond the Infinity Cache."""
    import numpy as np

    import gen

    p = gen.CONFIGS[name].params
    g = gen.make_graph(name, progress=log)
    kb = padded(p.k_block, p.dtype)
    col = np.asarray(g.col, np.int32)
    rng = np.random.default_rng(1)
    row_bytes = kb * elem_bytes(p.dtype)
    streams = {"spmm_column_indices": (col, g.n)}
    for F in (1 << 14, 1 << 17, 1 << 19, 1 << 20):
        streams[f"folded_{F * row_bytes >> 20}MiB"] = ((col % F).astype(np.int32), F)
    streams["shuffled"] = (rng.permutation(col), g.n)
    streams["sorted"] = (np.sort(col), g.n)
    streams["hub_ids_below_131072"] = (col[col < 131072], g.n)
    streams["ids_from_131072"] = (col[col >= 131072], g.n)
    for R in (g.n, 8 << 20, 16 << 20):
        streams[f"uniform_{R * row_bytes >> 20}MiB"] = (
            rng.integers(0, R, size=col.size, dtype=np.int32), R)
    res = gather_ceiling(g, kb, p.dtype, torch, streams=streams)
    return {"table": "gather_ceiling", "workload": name, "row_bytes": row_bytes,
            "indices": int(col.size), "kernel": "k_probe_gather", "rows": res}


def gather_slices(name: str, torch, reps: int = 5):
    """The gather probe on the workload's own column indices with each p row split into
    S column slices gathered by separate blocks (block b takes slice b % S, so each XCD's
    L2 holds one slice of the rows: erc_probe_gather_sliced), for every S that keeps a
    slice at 64 bytes or more.  Median of `reps` launches after a warm-up, HIP events;
    the rate counts the whole row (all slices) per index."""
    import numpy as np

    import gen
    from paper_2609_27209_amd import _abi

    p = gen.CONFIGS[name].params
    g = gen.make_graph(name, progress=log)
    kb = padded(p.k_block, p.dtype)
    full = kb * elem_bytes(p.dtype)
    idx = torch.from_numpy(np.ascontiguousarray(g.col, np.int32)).cuda()
    table = torch.empty(g.n * full // 4, dtype=torch.float32, device="cuda")
    table.uniform_()
    st = torch.cuda.current_stream()
    rows = {}
    S = 1
    while full // S >= 64 and S <= 8:
        rb = full // S
        out = torch.empty(S * _abi.erc_probe_out_bytes(idx.numel(), rb) // 4,
                          dtype=torch.float32, device="cuda")
        ts = []
        for r in range(reps + 1):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(st)
            _abi.erc_probe_gather_sliced(idx.data_ptr(), idx.numel(), table.data_ptr(), g.n, rb,
                                         S, out.data_ptr(), st.cuda_stream)
            e1.record(st)
            torch.cuda.synchronize()
            if r > 0:
                ts.append(e0.elapsed_time(e1))
        ms = sorted(ts)[len(ts) // 2]
        rows[str(S)] = {"slice_bytes": rb, "ms": round(ms, 4),
                        "gathered_gbs": round(idx.numel() * full / (ms / 1e3) / 1e9, 1),
                        "per_xcd_footprint_bytes": g.n * rb}
        log(f"sliced gather {name} S={S}: {rows[str(S)]}")
        del out
        S *= 2
    return {"table": "gather_slices", "workload": name, "row_bytes": full,
            "indices": int(idx.numel()), "kernel": "k_probe_gather", "rows": rows}


def _kernel_label(name: str) -> str:
    """Short kernel name of a rocprofv3 record (the template arguments kept)."""
    import re

    m = re.search(r"(k_\w+<[^>]*>|k_\w+|__amd\w+|\w*elementwise\w*)", name)
    return m.group(1) if m else name[:60]


def trace_table(path: str, full_us: float = 20.0, min_ms: float = 0.0) -> str:
    """Markdown table of a rocprofv3 kernel trace (its *_kernel_trace.csv): dispatches,
    total and average duration per kernel, and the average over "full" dispatches (those
    longer than full_us; launches after the last column converged return at once)."""
    import collections
    import csv

    d = collections.defaultdict(list)
    with open(path) as f:
        for r in csv.DictReader(f):
            d[_kernel_label(r["Kernel_Name"])].append(
                int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    tot = sum(sum(v) for v in d.values())
    out = ["| kernel | dispatches | total ms | avg us (all) | avg us (> 20 us) | full | share |",
           "|---|---|---|---|---|---|---|"]
    for k, v in sorted(d.items(), key=lambda kv: -sum(kv[1])):
        if sum(v) / 1e6 < min_ms:
            continue
        full = [x for x in v if x > full_us * 1e3]
        avgf = sum(full) / len(full) / 1e3 if full else 0.0
        out.append(f"| {k} | {len(v)} | {sum(v) / 1e6:.1f} | {sum(v) / len(v) / 1e3:.1f} | "
                   f"{avgf:.1f} | {len(full)} | {100 * sum(v) / tot:.1f}% |")
    return "\n".join(out)


def counter_table(path: str, full_us: float = 20.0) -> str:
    """Per kernel of a rocprofv3 counter run (its *_counter_collection.csv): dispatches,
    full dispatches and the median counter value over the full ones."""
    import collections
    import csv
    import statistics

    d = collections.defaultdict(list)
    with open(path) as f:
        for r in csv.DictReader(f):
            d[(_kernel_label(r["Kernel_Name"]), r["Counter_Name"])].append(
                (float(r["Counter_Value"]), int(r["End_Timestamp"]) - int(r["Start_Timestamp"])))
    out = ["| kernel | counter | dispatches | full | median (full) |", "|---|---|---|---|---|"]
    for (k, c), v in d.items():
        full = [x for x, dur in v if dur > full_us * 1e3]
        med = f"{statistics.median(full):.1f}" if full else "-"
        out.append(f"| {k} | {c} | {len(v)} | {len(full)} | {med} |")
    return "\n".join(out)


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="cl2400k")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-scale", type=int, default=25,
                    help="the CPU baseline runs on a 1/cpu-scale instance of the workload")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the Jacobi-preconditioned variant after the timed steps")
    ap.add_argument("--configs", action="store_true",
                    help="instead of the benchmark line: one line with every workload's "
                         "edges/s, iterations, SpMM time and device memory per block width")
    ap.add_argument("--only", default=None, metavar="NAME,NAME,...",
                    help="with --configs: only these workloads")
    ap.add_argument("--block-sweep", default=None, metavar="B,B,...",
                    help="instead of the benchmark line: one line with the --config "
                         "workload's step time, iterations and device memory at each of "
                         "these block widths")
    ap.add_argument("--no-draw", action="store_true",
                    help="skip the subgraph-draw measurement after the timed steps")
    ap.add_argument("--no-relabel", action="store_true",
                    help="skip the step on a randomly relabelled copy of the graph")
    ap.add_argument("--no-gather-probe", action="store_true",
                    help="skip timing the gather probe on the SpMM's column indices")
    ap.add_argument("--gather-ceiling", action="store_true",
                    help="instead of the benchmark line: one line with the gather probe's "
                         "rate on the --config workload's column indices and on index "
                         "streams with controlled footprints")
    ap.add_argument("--gather-slices", action="store_true",
                    help="instead of the benchmark line: one line with the gather probe's "
                         "rate on the --config workload's column indices with each row "
                         "gathered in 1, 2, 4 or 8 column slices by separate blocks")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after the timed steps, copy a buffer of this size 3 times (a plain "
                         "copy kernel of known size, to calibrate HBM byte counters)")
    ap.add_argument("--trace-table", default=None, metavar="CSV",
                    help="print the per-kernel table of a rocprofv3 kernel trace "
                         "(*_kernel_trace.csv) and exit (no GPU needed)")
    ap.add_argument("--counter-table", action="append", default=None, metavar="CSV",
                    help="print the per-kernel median counter values of a rocprofv3 --pmc "
                         "run (*_counter_collection.csv; may be given more than once) and "
                         "exit (no GPU needed)")
    ap.add_argument("--table-min-ms", type=float, default=0.0,
                    help="with --trace-table: list only kernels with at least this many ms")
    args = ap.parse_args()
    if args.trace_table or args.counter_table:
        if args.trace_table:
            print(trace_table(args.trace_table, min_ms=args.table_min_ms))
        for path in args.counter_table or []:
            print(counter_table(path))
        return 0
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the column "
              "sharding over several GPUs (a range of columns per GPU, then one sum of R) "
              "is not built.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import gen
    import paper_2609_27209_amd as E

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    torch.cuda.set_device(0)
    if args.configs:
        only = set(args.only.split(",")) if args.only else None
        print(json.dumps(per_config_table(args.steps, args.warmup, only)), flush=True)
        return 0
    if args.block_sweep:
        widths = [int(b) for b in args.block_sweep.split(",")]
        print(json.dumps(block_sweep(args.config, widths)), flush=True)
        return 0
    if args.gather_ceiling:
        print(json.dumps(gather_footprints(args.config, torch)), flush=True)
        return 0
    if args.gather_slices:
        print(json.dumps(gather_slices(args.config, torch)), flush=True)
        return 0
    wl = gen.CONFIGS[args.config]
    p = wl.params
    t0 = time.perf_counter()
    g = gen.make_graph(args.config, progress=log)
    log(f"graph {args.config}: {g.summary()} ({time.perf_counter() - t0:.1f}s)")
    t0 = time.perf_counter()
    G = E.Graph(g.rowptr, g.col, g.w, solve_dtype=p.dtype)
    torch.cuda.synchronize()
    log(f"erc_create {time.perf_counter() - t0:.1f}s")

    last = {}

    def step(profile: bool):
        R, info = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed,
                               profile=profile)
        pp, kk = G.curvature(R)
        pn, pe = G.sampling_probs(kk, p.eta)
        last["R"], last["pn"], last["pe"] = R, pn, pe
        return info

    for i in range(args.warmup):
        t = time.perf_counter()
        info = step(False)
        torch.cuda.synchronize()
        log(f"warmup {i}: {time.perf_counter() - t:.3f}s iters_max {info['iters_max']}")

    infos = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    step_ms = []
    for i in range(args.steps):
        ts = time.perf_counter()
        infos.append(step(True))
        torch.cuda.synchronize()  # a step is seconds long; this adds microseconds
        step_ms.append((time.perf_counter() - ts) * 1000.0)
        log(f"step {i}: {step_ms[-1]:.1f} ms, iters_max {infos[-1]['iters_max']} "
            f"cg {infos[-1]['ms_cg']:.1f}ms")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed * 1000.0 / args.steps
    value = g.m / (ms_per_step / 1000.0)

    kb = padded(p.k_block, p.dtype)
    # every SpMM launch is bracketed by HIP events on the solve stream; launches that
    # found no active column (issued before the host saw convergence) return at once,
    # so the average is taken over the full launches
    spmm_ms = sum(i["ms_spmm"] for i in infos)
    spmm_full = sum(i["spmm_full"] for i in infos)
    spmm_n = sum(i["spmm_timed"] for i in infos)
    avg_spmm_ms = spmm_ms / max(spmm_full, 1)
    bytes_launch = spmm_bytes_per_launch(g, kb, p.dtype)
    fused_launch = spmm_fused_bytes_per_launch(g, kb, p.dtype)
    achieved = bytes_launch / (avg_spmm_ms / 1000.0) / 1e9
    traffic = None
    if (MEASURED_TRAFFIC["workload"] == args.config
            and MEASURED_TRAFFIC["source_sha256_16"] == kernel_source_hash()):
        traffic = MEASURED_TRAFFIC["fetch_bytes"] + MEASURED_TRAFFIC["write_bytes"]
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic,
                "kernel": "k_spmm", "bytes_per_launch": bytes_launch,
                "avg_launch_ms": round(avg_spmm_ms, 4), "launches_full": spmm_full,
                "launches_timed": spmm_n,
                "fused_bytes_per_launch": fused_launch,
                "achieved_on_fused_bytes": round(fused_launch / (avg_spmm_ms / 1e3) / 1e9, 1)}
    if traffic is not None:
        tb = traffic / (avg_spmm_ms / 1000.0) / 1e9
        # L2-to-fabric rate: requests served by the Infinity Cache count as well as HBM
        roofline["fabric_gbs"] = round(tb, 1)
        roofline["fabric_vs_hbm_peak"] = round(tb / PEAK_HBM_GBS, 4)
        roofline["traffic_counted"] = "FETCH_SIZE + WRITE_SIZE: L2-to-fabric bytes (HBM and Infinity Cache)"
    iters_total = infos[-1]["iters_total"]
    # the whole CG inner loop (SpMM + finishing step + update) on the model bytes of an
    # iteration, over the timed steps
    ib = iteration_bytes(g, kb, p.dtype)
    ms_cg = sum(i["ms_cg"] for i in infos)
    loop_gbs = ib * spmm_full / (ms_cg / 1e3) / 1e9
    roofline["inner_loop"] = {"bytes_per_iteration": ib, "iterations": spmm_full,
                              "ms": round(ms_cg, 1), "achieved": round(loop_gbs, 1),
                              "frac": round(loop_gbs / PEAK_HBM_GBS, 4)}
    if not args.no_gather_probe:
        gc = gather_ceiling(g, kb, p.dtype, torch)["spmm_column_indices"]
        roofline["gather_ceiling"] = dict(gc, kernel="k_probe_gather",
                                          spmm_time_over_probe=round(avg_spmm_ms / gc["ms"], 3))

    draw = None if args.no_draw else subgraph_draw(G, last["pn"], last["pe"], torch)
    variants = None if args.no_variants else {"jacobi": jacobi_variant(G, g, p, last["R"], torch)}
    relabelled = None
    if not args.no_relabel:
        G.close()
        del G
        last.clear()
        torch.cuda.empty_cache()
        relabelled = relabelled_step(g, p, torch)

    if args.copy_probe_mib > 0:
        nb = args.copy_probe_mib << 20
        src = torch.ones(nb // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)  # an elementwise kernel: reads nb bytes, writes nb
        torch.cuda.synchronize()
        log(f"copy probe: 3 x {nb} bytes read + written")
        del src, dst

    cpu = None
    if not args.no_cpu_baseline:
        try:
            cpu = cpu_baseline(g, p, wl, iters_total, args.cpu_scale)
        except MemoryError as exc:  # pragma: no cover - host-dependent
            log(f"cpu baseline skipped: {exc}")

    summ = g.summary()
    line = {
        "metric": "CG SpMM achieved HBM GB/s (% peak) + curvature edges/sec end-to-end",
        "value": value,
        "unit": "edges/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "ms_per_step_median": round(sorted(step_ms)[len(step_ms) // 2], 2),
        "step_ms": [round(t, 2) for t in step_ms],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if p.dtype == "f32" else "f64",
        "data": "synthetic",
        "config": {"workload": args.config, "description": wl.description, "n": g.n, "m": g.m,
                   "deg_min": summ["deg_min"], "deg_median": summ["deg_median"],
                   "deg_max": summ["deg_max"], "components": gen.component_count(g),
                   "K": p.K, "k_block": p.k_block, "delta": p.delta, "tol": p.tol,
                   "seed": p.seed, "parallelism": "single GPU"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "subgraph_draw": draw,
        "variants": variants,
        "relabelled_copy": relabelled,
        "solve": {"iters_max": infos[-1]["iters_max"], "iters_total": iters_total,
                  "max_final_relres": infos[-1]["max_final_relres"],
                  "ms_rhs": infos[-1]["ms_rhs"], "ms_cg": infos[-1]["ms_cg"],
                  "ms_accum": infos[-1]["ms_accum"],
                  "bytes_model": infos[-1]["bytes_model"],
                  "model_gbs": round(infos[-1]["bytes_model"] / (infos[-1]["ms_total"] / 1e3)
                                     / 1e9, 1),
                  "edge_columns_per_s": g.m * p.K / (ms_per_step / 1000.0)},
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())

"""Curvature-agreement study of Section 4 (Table 2) with the GPU path as ERC-LG.

ERC-REG (dense (L + delta I)^-1), ERC-JL (the same JL sketch, dense direct solve) and
the pseudoinverse reference come from the oracle's stored values in
tests/golden/sbm2k_agreement.npz; ERC-LG runs erc_resistance + erc_curvature on the
GPU for each K.  Each method is scored against the pseudoinverse curvature by MAE,
Spearman correlation and sign agreement.

    python tests/agreement_study.py [out.json]
"""
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import gen  # noqa: E402
from oracle import agreement as AG  # noqa: E402

GOLDEN = os.path.join(ROOT, "tests", "golden", "sbm2k_agreement.npz")


def load_golden():
    with np.load(GOLDEN) as f:
        meta = json.loads(str(f["meta"]))
        return meta, {k: f[k] for k in f.files if k != "meta"}


def run_lg(G, K, params):
    """ERC-LG on the GPU: R over all K columns, then the curvature; host arrays."""
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    R, info = G.resistance(K, params.k_block, params.delta, params.tol, params.max_iter,
                           params.seed)
    _, kappa = G.curvature(R)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3
    return R.cpu().numpy(), kappa.cpu().numpy(), info, ms


def study():
    import paper_2609_27209_amd as E
    meta, gold = load_golden()
    wl = gen.CONFIGS["sbm2k"]
    g = gen.make_graph("sbm2k")
    G = E.Graph(g.rowptr, g.col, g.w, wl.params.dtype)
    kp = gold["kappa_pinv"]
    rows = [{"K": None, "method": "ERC-REG", **AG.metrics(gold["kappa_reg"], kp)}]
    lg = {}
    for K in meta["Ks"]:
        R, kappa, info, ms = run_lg(G, K, wl.params)
        lg[K] = (R, kappa, info)
        rows.append({"K": K, "method": "ERC-JL", **AG.metrics(gold[f"kappa_jl_{K}"], kp)})
        rows.append({"K": K, "method": "ERC-LG", **AG.metrics(kappa, kp), "ms": ms,
                     "blocks": info["blocks"], "iters_max": info["iters_max"]})
    return meta, gold, rows, lg


def format_table(rows):
    out = ["| K | method | MAE | Spearman | Sign | GPU ms |", "|---|---|---|---|---|---|"]
    for r in rows:
        ms = f"{r['ms']:.0f}" if "ms" in r else ""
        out.append(f"| {r['K'] or '-'} | {r['method']} | {r['mae']:.5f} | {r['spearman']:.4f} "
                   f"| {r['sign']:.4f} | {ms} |")
    return "\n".join(out)


if __name__ == "__main__":
    meta, gold, rows, lg = study()
    print(format_table(rows), flush=True)
    if len(sys.argv) > 1:
        with open(sys.argv[1], "w") as f:
            json.dump({"graph": meta["graph"], "rows": rows}, f, indent=1)

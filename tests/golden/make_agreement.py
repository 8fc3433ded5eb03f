"""Write the stored oracle curvatures of the agreement study (Table 2 of Section 4).

    python tests/golden/make_agreement.py

On the SBM workload sbm2k it computes, with oracle/ only, the edge curvature from
the pseudoinverse resistance (Eq. 1), from the diagonal-perturbation resistance
b^T (L + delta I)^{-1} b (ERC-REG) and from the JL estimate with a dense direct
solve of Eq. 5 (ERC-JL) for K = 1024, 2048 and 4096, all sketches using the
projection seed of the workload, and stores them in tests/golden/sbm2k_agreement.npz.
"""
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import gen  # noqa: E402
from oracle import agreement as AG  # noqa: E402
from oracle import erc as OE  # noqa: E402
from oracle import exact as EX  # noqa: E402

KS = (1024, 2048, 4096)


def main():
    wl = gen.CONFIGS["sbm2k"]
    p = wl.params
    g = gen.make_graph("sbm2k")
    out = {}
    t0 = time.time()
    _, out["kappa_pinv"] = OE.curvature(g, EX.pinv_resistance(g))
    _, out["kappa_reg"] = OE.curvature(g, EX.reg_resistance(g, p.delta))
    table = {"REG": AG.metrics(out["kappa_reg"], out["kappa_pinv"])}
    for K in KS:
        R = EX.jl_dense_resistance(g, K, p.seed, p.delta)
        out[f"R_jl_{K}"] = R
        _, out[f"kappa_jl_{K}"] = OE.curvature(g, R)
        table[f"JL{K}"] = AG.metrics(out[f"kappa_jl_{K}"], out["kappa_pinv"])
        print(f"[agreement] K={K} {table[f'JL{K}']} ({time.time() - t0:.0f}s)", flush=True)
    meta = {"workload": "sbm2k", "graph": g.summary(), "delta": p.delta, "seed": p.seed,
            "Ks": list(KS), "oracle_metrics": table}
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "sbm2k_agreement.npz")
    np.savez_compressed(path, meta=np.array(json.dumps(meta)), **out)
    print(f"[agreement] wrote {path}", flush=True)


if __name__ == "__main__":
    main()

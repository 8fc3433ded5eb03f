"""Write SHA-256 digests of the oracle's edge numbering and right-hand sides.

    python tests/golden/make_digests.py [workload ...]

For each workload (default: all five performance workloads) this regenerates the
seeded graph and hashes, with the CPU oracle only (gen/ and oracle/, nothing from the
GPU library):

* the canonical edge id of every stored CSR entry, as little-endian int32 (the
  edge numbering of Section 3.1.1: edge e is the e-th pair u < v in lexicographic
  order), and the edge list's endpoints u and v, as little-endian int32;
* the right-hand sides Y = B^T W^{1/2} Q of Section 3.1.2 for the column blocks in
  BLOCKS, in the workload's working precision, row-major n x ncols, little-endian.

The GPU test hashes erc_debug_edge_ids, erc_edge_endpoints and erc_debug_rhs output
at the same sizes and compares: every bit of the indexing, the signs and the values
must agree.  Digests go to tests/golden/digests.json (merged with what is there).
"""
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import gen  # noqa: E402
from oracle import erc as OE  # noqa: E402
from oracle import graph as OG  # noqa: E402

# (col0, ncols) per workload: the whole sketch where it is one block, else the first
# block, and on the 2.4M-node graph also the last block (sign word 3)
BLOCKS = {
    "er2k": [(0, 32)],
    "sbm20k": [(0, 64)],
    "cl170k": [(0, 128)],
    "cl230k": [(0, 32), (96, 32)],
    "cl2400k": [(0, 64), (192, 64)],
}
OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "digests.json")


def sha(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def log(msg):
    print(f"[digests] {msg}", flush=True)


def make(name):
    p = gen.CONFIGS[name].params
    g = gen.make_graph(name, progress=log)
    eu, ev, eid = OG.canonical_edges(g)
    rec = {"graph": g.summary(), "K": p.K, "seed": p.seed, "dtype": p.dtype,
           "eid_int32": sha(eid.astype("<i4")), "eu_int32": sha(eu.astype("<i4")),
           "ev_int32": sha(ev.astype("<i4")), "rhs": []}
    wdt = "<f4" if p.dtype == "f32" else "<f8"
    for col0, ncols in BLOCKS[name]:
        t0 = time.time()
        Y = OE.rhs(g, p.K, col0, ncols, p.seed, p.dtype)
        rec["rhs"].append({"col0": col0, "ncols": ncols, "sha256": sha(Y.astype(wdt))})
        log(f"{name}: rhs [{col0}, {col0 + ncols}) in {time.time() - t0:.0f}s")
    return rec


def main(names):
    data = {}
    if os.path.exists(OUT):
        with open(OUT) as f:
            data = json.load(f)
    for name in names:
        data[name] = make(name)
        with open(OUT, "w") as f:
            json.dump(data, f, indent=1, sort_keys=True)
        log(f"wrote {name} to {OUT}")


if __name__ == "__main__":
    main(sys.argv[1:] or list(BLOCKS))

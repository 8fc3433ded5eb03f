"""Bit-exact edge numbering and right-hand sides at every workload size.

tests/golden/digests.json holds SHA-256 digests written by
tests/golden/make_digests.py from the CPU oracle alone: the canonical edge id of every
stored CSR entry and the edge list's endpoints (Section 3.1.1), and the right-hand
sides Y = B^T W^{1/2} Q of Section 3.1.2 for whole column blocks, in the working
precision.  The GPU's erc_debug_edge_ids, erc_edge_endpoints and erc_debug_rhs output
is hashed the same way; equal digests mean every index, sign and value bit agrees.
"""
import hashlib
import json
import os

import numpy as np
import pytest

import gen

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

DIGESTS = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "digests.json")


def _sha(t) -> str:
    return hashlib.sha256(np.ascontiguousarray(t.cpu().numpy()).tobytes()).hexdigest()


def _load():
    with open(DIGESTS) as f:
        return json.load(f)


@pytest.mark.parametrize("name", ["er2k", "sbm20k", "cl170k", "cl230k", "cl2400k"])
def test_indexing_and_rhs_digests(name):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_27209_amd as E

    rec = _load()[name]
    p = gen.CONFIGS[name].params
    assert (rec["K"], rec["seed"], rec["dtype"]) == (p.K, p.seed, p.dtype)
    g = gen.make_graph(name)
    assert g.summary() == rec["graph"], "generator output differs from the hashed graph"
    G = E.Graph(g.rowptr, g.col, g.w, solve_dtype=p.dtype)
    eid = G.debug_edge_ids()
    u, v = G.edge_endpoints()
    torch.cuda.synchronize()
    assert _sha(eid) == rec["eid_int32"], f"{name}: edge ids differ"
    assert _sha(u) == rec["eu_int32"] and _sha(v) == rec["ev_int32"], f"{name}: endpoints differ"
    for blk in rec["rhs"]:
        Y = G.debug_rhs(p.K, blk["col0"], blk["ncols"], p.seed)
        torch.cuda.synchronize()
        assert Y.dtype == (torch.float32 if p.dtype == "f32" else torch.float64)
        assert _sha(Y) == blk["sha256"], f"{name}: RHS columns [{blk['col0']}, " \
            f"{blk['col0'] + blk['ncols']}) differ"
        print(f"{name}: RHS [{blk['col0']}, {blk['col0'] + blk['ncols']}) bit-exact", flush=True)
        del Y
    G.close()

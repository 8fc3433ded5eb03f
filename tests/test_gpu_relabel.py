"""GPU parity on a randomly relabelled copy of a power-law workload.

The Chung-Lu generator numbers nodes in decreasing expected degree, so the hub rows sit
at the front of every array and the SpMM's work plan meets them first.  A caller's graph
need not be ordered that way.  These tests run the path on the 170k-node workload with
its node ids randomly permuted (same structure, degrees and weights; the hubs scattered
over the id range) against the CPU oracle on the same relabelled graph and seeds: edge
ids and right-hand sides bit for bit (Section 3.1.2) and the operator of Eq. 5.  The
resistance, curvature and sampling probabilities of the same relabelled copy are
compared with stored oracle values in test_gpu_large.py (cl170k_relabel).
"""
import numpy as np
import pytest

import gen
from oracle import erc as OE
from oracle import graph as OG

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

NAME = "cl170k"


@pytest.fixture(scope="module")
def relabelled():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_27209_amd as E

    g0 = gen.make_graph(NAME)
    perm = np.random.default_rng(7).permutation(g0.n)
    g = gen.relabel(g0, perm)
    # node perm[i] of the copy has node i's degree: the hubs no longer lead
    assert np.array_equal(np.diff(g.rowptr)[perm], np.diff(g0.rowptr))
    p = gen.CONFIGS[NAME].params
    G = E.Graph(g.rowptr, g.col, g.w, solve_dtype=p.dtype)
    return E, g, p, G


def test_relabelled_edge_ids_and_rhs_bit_exact(relabelled):
    E, g, p, G = relabelled
    _, _, eid = OG.canonical_edges(g)
    assert np.array_equal(G.debug_edge_ids().cpu().numpy(), eid)
    Y = G.debug_rhs(p.K, 0, p.k_block, p.seed).cpu().numpy()
    Yo = OE.rhs(g, p.K, 0, p.k_block, p.seed, p.dtype)
    assert Y.dtype == Yo.dtype and np.array_equal(Y.view(np.uint8), Yo.view(np.uint8))


def test_relabelled_operator(relabelled):
    E, g, p, G = relabelled
    X = np.random.default_rng(3).standard_normal((g.n, p.k_block)).astype(np.float32)
    Yg = G.debug_spmm(p.delta, torch.from_numpy(X)).cpu().numpy().astype(np.float64)
    L = OG.laplacian(g)
    X64 = X.astype(np.float64)
    Yo = OE.laplacian_apply(L, p.delta, X64)
    # fp32 rounding bound: 4 u (deg + 2) (sum_j w_ij (|x_i| + |x_j|) + delta |x_i|)
    scale = abs(L) @ np.abs(X64) + p.delta * np.abs(X64)
    deg = np.diff(g.rowptr)[:, None] + 2
    assert np.all(np.abs(Yg - Yo) <= 4 * 2.0 ** -24 * deg * scale + 1e-300)

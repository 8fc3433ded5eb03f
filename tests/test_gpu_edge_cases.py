"""GPU edge cases of the whole path against the oracle: graphs without edges (every
right-hand side is zero, so every column converges at iteration 0; p = 1 and no node
has a positive sampling weight), a graph of one node, and the widest blocks in both
precisions on a graph with a ragged last block."""
import numpy as np
import pytest

import gen
from oracle import erc as OE
from oracle import sampling as OS

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_27209_amd as E
    return E


@pytest.mark.parametrize("n", [1, 7])
@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_edgeless_graph(n, dtype):
    E = _gpu()
    from paper_2609_27209_amd import _abi
    g = gen.from_edges(n, [], [])
    G = E.Graph(g.rowptr, g.col, g.w, dtype)
    assert (G.n, G.m) == (n, 0)
    R, info = G.resistance(16, 16, 1e-5, 1e-6, 100, 3)
    assert R.numel() == 0
    assert info["iters_max"] == 0 and info["cols_unconverged"] == 0 and info["breakdowns"] == 0
    p, kappa = G.curvature(R)
    assert kappa.numel() == 0
    np.testing.assert_array_equal(p.cpu().numpy(), np.ones(n))
    pn, pe = G.sampling_probs(kappa, 1e-12)
    ref_pn, ref_pe = OE.sampling_probs(g, np.zeros(0), 1e-12)
    np.testing.assert_array_equal(pn.cpu().numpy(), ref_pn)
    assert pe.numel() == 0
    u, v = G.edge_endpoints()
    assert u.numel() == 0 and v.numel() == 0
    with pytest.raises(_abi.ErcError) as ei:
        G.draw("nodes", pn, 10, 1)        # every weight is zero
    assert ei.value.status == _abi.ERC_E_NUMERIC
    with pytest.raises(_abi.ErcError) as ei:
        G.draw("edges", pe, 10, 1)        # nothing to draw from
    assert ei.value.status == _abi.ERC_E_INVALID_ARG
    idx = torch.tensor([0, n - 1, 0], dtype=torch.int64, device="cuda")
    sg = G.subgraph("nodes", idx)
    ref = OS.node_subgraph(g, idx.cpu().numpy())
    np.testing.assert_array_equal(sg["nodes"].cpu().numpy(), ref["nodes"])
    assert sg["edges"].numel() == 0


@pytest.mark.parametrize("dtype,kb,K", [("f32", 256, 300), ("f64", 128, 150)])
def test_widest_blocks_with_ragged_tail(dtype, kb, K):
    # two blocks: one full block of the widest width and a ragged one
    E = _gpu()
    g = gen.erdos_renyi(500, 0.02, 11, weighted=True)
    G = E.Graph(g.rowptr, g.col, g.w, dtype)
    R, info = G.resistance(K, kb, 1e-5, 1e-9 if dtype == "f64" else 1e-6, 5000, 21)
    assert info["blocks"] == 2 and info["cols_unconverged"] == 0
    ref, _ = OE.resistance(g, K, kb, 1e-5, 1e-9 if dtype == "f64" else 1e-6, 5000, 21, dtype)
    rel = np.max(np.abs(R.cpu().numpy() - ref) / ref)
    assert rel <= (1e-9 if dtype == "f64" else 1e-4), rel

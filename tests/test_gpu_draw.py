"""GPU parity of the curvature-guided subgraph draw (erc_draw, erc_subgraph) against the
oracle's definition (oracle/sampling.py): draws and subgraphs are integer results and
must match bit for bit on the same probabilities and seed.  The probabilities come from
the oracle's Eqs. 7-8 on seeded resistances, so nothing here depends on the solve."""
import numpy as np
import pytest
from scipy import stats

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


def _probs(g, seed=0):
    R = np.random.default_rng(seed).random(g.m) * 2.0 + 0.05
    _, kappa = OE.curvature(g, R)
    return OE.sampling_probs(g, kappa, 1e-12)


def _dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


GRAPHS = {
    "er2k": lambda: gen.make_graph("er2k"),
    "sbm20k": lambda: gen.make_graph("sbm20k"),
    # 3 tiles of 4096 items and a ragged tail, as nodes and as edges
    "path12305": lambda: gen.path_graph(3 * 4096 + 17),
    "isolated": lambda: gen.from_edges(9, [0, 1, 2, 4, 5], [1, 2, 0, 5, 6]),
}


@pytest.mark.parametrize("name", sorted(GRAPHS))
@pytest.mark.parametrize("items", ["nodes", "edges"])
def test_draw_bit_exact(name, items):
    E = _gpu()
    g = GRAPHS[name]()
    pn, pe = _probs(g, 1)
    P = pn if items == "nodes" else pe
    G = E.Graph(g.rowptr, g.col, g.w)
    got = G.draw(items, _dev(P), 20000, seed=31).cpu().numpy()
    np.testing.assert_array_equal(got, OS.draw(P, 20000, 31))


def test_draw_many_tiles_cl170k_edges():
    # 1.23M edges: 301 scan tiles, so the block-sum scan runs over several chunks
    E = _gpu()
    g = gen.make_graph("cl170k")
    _, pe = _probs(g, 2)
    G = E.Graph(g.rowptr, g.col, g.w)
    got = G.draw("edges", _dev(pe), 5000, seed=8).cpu().numpy()
    np.testing.assert_array_equal(got, OS.draw(pe, 5000, 8))


def test_draw_point_mass_zero_weights_and_empty():
    E = _gpu()
    g = gen.path_graph(10)
    G = E.Graph(g.rowptr, g.col, g.w)
    P = np.zeros(10)
    P[6] = 1.0
    assert set(G.draw("nodes", _dev(P), 1000, 3).cpu().numpy().tolist()) == {6}
    P = np.array([0.25, 0, 0, 0.25, 0, 0, 0.5, 0, 0, 0])
    got = G.draw("nodes", _dev(P), 4000, 4).cpu().numpy()
    assert set(got.tolist()) <= {0, 3, 6}
    np.testing.assert_array_equal(got, OS.draw(P, 4000, 4))
    assert G.draw("nodes", _dev(P), 0, 4).numel() == 0


def test_draw_frequencies_chi_square():
    E = _gpu()
    g = gen.path_graph(60)
    rng = np.random.default_rng(3)
    P = rng.random(60) ** 2
    P[[5, 40]] = 0.0
    P /= P.sum()
    G = E.Graph(g.rowptr, g.col, g.w)
    n = 1_000_000
    cnt = np.bincount(G.draw("nodes", _dev(P), n, 99).cpu().numpy(), minlength=60)
    assert cnt[5] == 0 and cnt[40] == 0
    nz = P > 0
    chi2 = np.sum((cnt[nz] - n * P[nz]) ** 2 / (n * P[nz]))
    assert stats.chi2.sf(chi2, nz.sum() - 1) > 1e-4


def test_draw_seeds():
    E = _gpu()
    g = gen.make_graph("er2k")
    pn, _ = _probs(g, 4)
    G = E.Graph(g.rowptr, g.col, g.w)
    a = G.draw("nodes", _dev(pn), 500, 1).cpu().numpy()
    b = G.draw("nodes", _dev(pn), 500, 2).cpu().numpy()
    assert not np.array_equal(a, b)
    np.testing.assert_array_equal(a, G.draw("nodes", _dev(pn), 500, 1).cpu().numpy())


@pytest.mark.parametrize("bad", ["nan", "negative", "above_one", "sum_two", "all_zero",
                                 "underflow"])
def test_draw_rejects_invalid_probabilities(bad):
    E = _gpu()
    from paper_2609_27209_amd import _abi
    g = gen.path_graph(5000)
    G = E.Graph(g.rowptr, g.col, g.w)
    P = np.full(5000, 1.0 / 5000)
    if bad == "nan":
        P[4500] = np.nan
    elif bad == "negative":
        P[3] = -1e-3
    elif bad == "above_one":
        P[7] = 1.5
    elif bad == "sum_two":
        P *= 2.0
    elif bad == "all_zero":
        P[:] = 0.0
    elif bad == "underflow":
        P[:] = 2.0 ** -70   # every integer weight is 0
    with pytest.raises(_abi.ErcError) as ei:
        G.draw("nodes", _dev(P), 100, 1)
    assert ei.value.status == _abi.ERC_E_NUMERIC
    # the next valid call on the same handle is unaffected
    Pv = np.full(5000, 1.0 / 5000)
    np.testing.assert_array_equal(G.draw("nodes", _dev(Pv), 100, 1).cpu().numpy(),
                                  OS.draw(Pv, 100, 1))


@pytest.mark.parametrize("name", ["er2k", "sbm20k", "isolated", "path12305"])
@pytest.mark.parametrize("items", ["nodes", "edges"])
def test_subgraph_bit_exact(name, items):
    E = _gpu()
    g = GRAPHS[name]()
    pn, pe = _probs(g, 5)
    G = E.Graph(g.rowptr, g.col, g.w)
    P = pn if items == "nodes" else pe
    draws = max(1, min(3000, P.size // 2))
    idx = G.draw(items, _dev(P), draws, 17)
    sg = G.subgraph(items, idx)
    ref = (OS.node_subgraph if items == "nodes" else OS.edge_subgraph)(g, idx.cpu().numpy())
    for k in ("nodes", "edges", "u", "v"):
        np.testing.assert_array_equal(sg[k].cpu().numpy(), ref[k], err_msg=k)


def test_subgraph_everything_nothing_and_repeats():
    E = _gpu()
    g = gen.make_graph("sbm20k")
    G = E.Graph(g.rowptr, g.col, g.w)
    from oracle import graph as OG
    eu, ev, _ = OG.canonical_edges(g)
    # every node: the whole graph, edges in canonical order with their own endpoints
    sg = G.subgraph("nodes", torch.arange(g.n, device="cuda"))
    assert sg["nodes"].numel() == g.n and sg["edges"].numel() == g.m
    np.testing.assert_array_equal(sg["u"].cpu().numpy(), eu)
    np.testing.assert_array_equal(sg["v"].cpu().numpy(), ev)
    # nothing drawn
    sg = G.subgraph("edges", torch.empty(0, dtype=torch.int64, device="cuda"))
    assert sg["nodes"].numel() == 0 and sg["edges"].numel() == 0
    # one edge drawn many times
    sg = G.subgraph("edges", torch.full((100,), 7, dtype=torch.int64, device="cuda"))
    assert sg["edges"].cpu().tolist() == [7]
    assert sg["nodes"].cpu().tolist() == [int(eu[7]), int(ev[7])]
    assert sg["u"].cpu().tolist() == [0] and sg["v"].cpu().tolist() == [1]


@pytest.mark.parametrize("items", ["nodes", "edges"])
def test_subgraph_rejects_out_of_range(items):
    E = _gpu()
    from paper_2609_27209_amd import _abi
    g = gen.path_graph(100)
    G = E.Graph(g.rowptr, g.col, g.w)
    bad = 100 if items == "nodes" else 99
    for idx in ([1, 2, bad], [-1]):
        with pytest.raises(_abi.ErcError) as ei:
            G.subgraph(items, torch.tensor(idx, dtype=torch.int64, device="cuda"))
        assert ei.value.status == _abi.ERC_E_INVALID_ARG

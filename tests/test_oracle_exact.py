"""Pins of the oracle's graph layer and exact references against closed forms.

Eq. 1 (R = b^T L^+ b) and Eq. 2 (p, kappa) are evaluated with the oracle and checked
against textbook values: series/parallel resistances, Foster's theorem
(sum_e w_e R_e = n - #components), bridges (R = 1/w), and the resulting curvatures.
"""
import numpy as np
import pytest

import gen
from oracle import erc, exact
from oracle import graph as GR


def hand_graph():
    # edges (0,2), (1,2), (0,1), (2,3) given out of order
    return gen.from_edges(4, [0, 2, 1, 3], [2, 1, 0, 2], np.array([1.0, 2.0, 3.0, 4.0]))


def test_canonical_edges_hand_example():
    g = hand_graph()
    eu, ev, eid = GR.canonical_edges(g)
    assert eu.tolist() == [0, 0, 1, 2]
    assert ev.tolist() == [1, 2, 2, 3]
    # CSR rows: 0:[1,2]  1:[0,2]  2:[0,1,3]  3:[2]
    assert g.col.tolist() == [1, 2, 0, 2, 0, 1, 3, 2]
    assert eid.tolist() == [0, 1, 0, 2, 1, 2, 3, 3]
    # weights follow their edges: (0,2)=1, (1,2)=2, (0,1)=3, (2,3)=4
    assert GR.edge_weights(g).tolist() == [3.0, 1.0, 2.0, 4.0]


def test_incidence_orientation_hand_example():
    g = hand_graph()
    B = GR.incidence(g).toarray()
    expect = np.array([[1, -1, 0, 0], [1, 0, -1, 0], [0, 1, -1, 0], [0, 0, 1, -1]], float)
    assert np.array_equal(B, expect)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_laplacian_btwb_equals_d_minus_a(seed):
    g = gen.erdos_renyi(40, 0.2, seed, weighted=True)
    L = GR.laplacian(g).toarray()
    assert np.allclose(L, GR.dense_laplacian(g), rtol=0, atol=1e-13)
    assert np.allclose(L @ np.ones(g.n), 0, atol=1e-12)
    assert np.allclose(L, L.T)


def test_check_graph_rejects():
    # each bad input breaks exactly one rule, and the message names that rule
    good = gen.cycle_graph(5)
    GR.check_graph(good)
    bad_sym = gen.CSRGraph(3, np.array([0, 1, 1, 1]), np.array([1], dtype=np.int32))
    with pytest.raises(ValueError, match="symmetric"):
        GR.check_graph(bad_sym)
    # (0, 0), (0, 1), (1, 0): symmetric and ascending, with a self-loop
    loop = gen.CSRGraph(2, np.array([0, 2, 3]), np.array([0, 1, 0], dtype=np.int32))
    with pytest.raises(ValueError, match="self-loop"):
        GR.check_graph(loop)
    # (0, 1) and (1, 0) stored twice each: symmetric, with repeats
    repeat = gen.CSRGraph(2, np.array([0, 2, 4]), np.array([1, 1, 0, 0], dtype=np.int32))
    with pytest.raises(ValueError, match="ascending"):
        GR.check_graph(repeat)
    unsorted = gen.CSRGraph(3, np.array([0, 2, 3, 4]), np.array([2, 1, 0, 0], dtype=np.int32))
    with pytest.raises(ValueError, match="ascending"):
        GR.check_graph(unsorted)
    g = gen.path_graph(3, w=np.array([1.0, 2.0]))
    w = g.w.copy()
    w[0] = -1.0
    with pytest.raises(ValueError, match="positive"):
        GR.check_graph(gen.CSRGraph(g.n, g.rowptr, g.col, w))
    w = g.w.copy()
    w[0] = 5.0  # breaks w_ij == w_ji
    with pytest.raises(ValueError, match="symmetric"):
        GR.check_graph(gen.CSRGraph(g.n, g.rowptr, g.col, w))


# ---- Eq. 1 against closed forms -------------------------------------------------

@pytest.mark.parametrize("n", [3, 5, 8])
def test_complete_graph_resistance(n):
    R = exact.pinv_resistance(gen.complete_graph(n))
    assert np.allclose(R, 2.0 / n, rtol=1e-12)


@pytest.mark.parametrize("n", [3, 7, 12])
def test_cycle_resistance(n):
    R = exact.pinv_resistance(gen.cycle_graph(n))
    assert np.allclose(R, (n - 1) / n, rtol=1e-12)


@pytest.mark.parametrize("a,b", [(2, 3), (3, 3), (2, 5)])
def test_complete_bipartite_resistance(a, b):
    R = exact.pinv_resistance(gen.complete_bipartite(a, b))
    assert np.allclose(R, (a + b - 1) / (a * b), rtol=1e-12)


def test_tree_edges_are_inverse_weights():
    g = gen.random_tree(30, seed=4, weighted=True)
    R = exact.pinv_resistance(g)
    assert np.allclose(R, 1.0 / GR.edge_weights(g), rtol=1e-10)


def test_series_parallel_weighted():
    # two parallel paths between 0 and 3: 0-1-3 (w 1, 2) and 0-2-3 (w 4, 4)
    g = gen.from_edges(4, [0, 1, 0, 2], [1, 3, 2, 3], np.array([1.0, 2.0, 4.0, 4.0]))
    eu, ev, _ = GR.canonical_edges(g)
    R = exact.pinv_resistance(g)
    # effective resistance between 0 and 1: r01 = 1 in parallel with (1/2 + 1/4 + 1/4)
    r01 = 1.0 / (1.0 / 1.0 + 1.0 / 1.0)
    got = dict(zip(zip(eu.tolist(), ev.tolist()), R))
    assert np.isclose(got[(0, 1)], r01, rtol=1e-12)
    # between 0 and 2: 1/4 in parallel with (1 + 1/2 + 1/4)
    r02 = 1.0 / (4.0 + 1.0 / 1.75)
    assert np.isclose(got[(0, 2)], r02, rtol=1e-12)


def test_barbell_bridges():
    g = gen.barbell_graph(5, bridge_len=3, seed=9)
    R = exact.pinv_resistance(g)
    eu, ev, _ = GR.canonical_edges(g)
    w = GR.edge_weights(g)
    bridge = (eu >= 4) & (ev <= 7) & (ev - eu == 1)
    assert bridge.sum() == 3
    assert np.allclose(R[bridge], 1.0 / w[bridge], rtol=1e-10)


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_foster(seed):
    g = gen.erdos_renyi(60, 0.08, seed, weighted=True)
    c = GR.components(g)
    R = exact.pinv_resistance(g)
    assert np.isclose(np.sum(GR.edge_weights(g) * R), g.n - c, rtol=1e-10)


# ---- Eq. 2 against closed forms -------------------------------------------------

@pytest.mark.parametrize("n", [4, 7])
def test_curvature_complete(n):
    g = gen.complete_graph(n)
    p, k = erc.curvature(g, exact.pinv_resistance(g))
    assert np.allclose(p, 1.0 / n, rtol=1e-12)
    assert np.allclose(k, 2.0, rtol=1e-12)


@pytest.mark.parametrize("n", [5, 9])
def test_curvature_cycle(n):
    g = gen.cycle_graph(n)
    p, k = erc.curvature(g, exact.pinv_resistance(g))
    assert np.allclose(p, 1.0 / n, rtol=1e-12)
    assert np.allclose(k, 4.0 / (n - 1), rtol=1e-12)


def test_curvature_path():
    n = 6
    g = gen.path_graph(n)
    p, k = erc.curvature(g, exact.pinv_resistance(g))
    assert np.allclose(p, [0.5, 0, 0, 0, 0, 0.5], atol=1e-12)
    assert np.allclose(k, [1, 0, 0, 0, 1], atol=1e-12)


@pytest.mark.parametrize("n", [3, 6])
def test_curvature_star(n):
    g = gen.star_graph(n)
    p, k = erc.curvature(g, exact.pinv_resistance(g))
    assert np.isclose(p[0], (3 - n) / 2)
    assert np.allclose(p[1:], 0.5)
    assert np.allclose(k, 4 - n, atol=1e-12)


def test_curvature_complete_bipartite():
    a, b = 2, 4
    g = gen.complete_bipartite(a, b)
    p, k = erc.curvature(g, exact.pinv_resistance(g))
    r = (a + b - 1) / (a * b)
    pa = 1 - (a + b - 1) / (2 * a)
    pb = 1 - (a + b - 1) / (2 * b)
    assert np.allclose(p[:a], pa) and np.allclose(p[a:], pb)
    assert np.allclose(k, 2 * (pa + pb) / r)


def test_node_curvature_sums_to_components():
    # sum_u p_u = n - sum_e w_e R_e = #components (Foster)
    g = gen.erdos_renyi(50, 0.06, 5, weighted=True)
    p, _ = erc.curvature(g, exact.pinv_resistance(g))
    assert np.isclose(p.sum(), GR.components(g), rtol=1e-10)


def test_isolated_node_curvature_is_one():
    g = gen.from_edges(4, [0, 1], [1, 2])  # node 3 isolated
    p, k = erc.curvature(g, exact.pinv_resistance(g))
    assert p[3] == 1.0
    assert np.allclose(k, [1.0, 1.0])


# ---- ERC-REG (prior work) and ERC-JL ---------------------------------------------

def test_reg_resistance_converges_to_pinv():
    g = gen.erdos_renyi(80, 0.1, 3, weighted=True)
    R = exact.pinv_resistance(g)
    e1 = np.abs(exact.reg_resistance(g, 1e-4) - R).max()
    e2 = np.abs(exact.reg_resistance(g, 1e-6) - R).max()
    assert e2 < 1e-5
    assert e2 < e1 / 50  # bias is linear in eps


def test_jl_dense_unbiased_on_bridges():
    # a bridge carries the whole unit current, so every Q gives R = 1/w
    g = gen.barbell_graph(6, bridge_len=2, seed=2)
    Rj = exact.jl_dense_resistance(g, 16, seed=5, delta=1e-10)
    eu, ev, _ = GR.canonical_edges(g)
    w = GR.edge_weights(g)
    bridge = (ev - eu == 1) & (eu >= 5) & (ev <= 7)
    assert bridge.sum() == 2
    assert np.allclose(Rj[bridge], 1.0 / w[bridge], rtol=1e-7)

"""Pins of the oracle's subgraph draw: the integer inverse CDF against exact cases
(point masses, zero weights, two-point laws), frequency tests of the draws against
the probabilities they come from, the 128-bit target against an independent formula,
and subgraph assembly against brute force."""
import math

import numpy as np
import pytest
from scipy import stats

import gen
from oracle import erc as OE
from oracle import graph as GR
from oracle import hashing as H
from oracle import sampling as S


def test_integer_weights_exact():
    W = S.integer_weights([0.5, 0.25, 0.0, 2.0 ** -62, 1.0])
    assert [int(x) for x in W] == [1 << 61, 1 << 60, 0, 1, 1 << 62]
    with pytest.raises(ValueError):
        S.integer_weights([0.5, np.nan])
    with pytest.raises(ValueError):
        S.integer_weights([-0.1, 1.1])


def test_targets_uniform_bits():
    # t = floor(X T / 2^128) for T = 2^k is the top k bits of X = x_hi (when k <= 64)
    words = H.splitmix64(int(H.base(7)), 20)
    t = S.draw_targets(7, 1 << 20, 10)
    assert t == [int(words[2 * d]) >> 44 for d in range(10)]


def test_select_on_cdf_boundaries():
    # W = [0, 3, 0, 5]: C = [0, 0, 3, 3, 8]; a target equal to C_i selects item i (the
    # first with positive weight at that point), never a zero-weight item
    C = np.array([0, 0, 3, 3, 8], dtype=np.uint64)
    assert S.select(C, [0, 1, 2, 3, 4, 7]).tolist() == [1, 1, 1, 3, 3, 3]
    # large weights near the top of the 64-bit range
    big = np.array([0, 2**62, 2**62, 2**63 - 1], dtype=np.uint64)
    assert S.select(big, [0, 2**62 - 1, 2**62, 2**63 - 2]).tolist() == [0, 0, 2, 2]


def test_point_mass_and_zero_weights():
    assert set(S.draw([0.0, 1.0, 0.0], 200, 3)) == {1}
    d = S.draw([0.5, 0.0, 0.5, 0.0], 2000, 4)
    assert set(d) <= {0, 2}
    assert abs(np.mean(d == 0) - 0.5) < 4 * math.sqrt(0.25 / 2000)


def test_draw_frequencies_chi_square():
    rng = np.random.default_rng(5)
    P = rng.random(40) ** 3
    P[7] = 0.0
    P /= P.sum()
    n = 40000
    d = S.draw(P, n, 11)
    cnt = np.bincount(d, minlength=P.size)
    assert cnt[7] == 0
    nz = P > 0
    chi2 = np.sum((cnt[nz] - n * P[nz]) ** 2 / (n * P[nz]))
    # p-value of the statistic with nz-1 degrees of freedom; a shifted CDF search
    # (an off-by-one) sends this to ~0
    assert stats.chi2.sf(chi2, nz.sum() - 1) > 1e-3


def test_different_seeds_differ_and_same_seed_repeats():
    P = np.full(1000, 1e-3)
    a, b = S.draw(P, 100, 1), S.draw(P, 100, 2)
    assert not np.array_equal(a, b)
    np.testing.assert_array_equal(a, S.draw(P, 100, 1))


def brute_subgraph(g, nodes=None, edges=None):
    eu, ev, _ = GR.canonical_edges(g)
    E = list(zip(eu.tolist(), ev.tolist()))
    if nodes is not None:
        V = sorted(set(int(x) for x in nodes))
        sel = [e for e, (u, v) in enumerate(E) if u in V and v in V]
    else:
        sel = sorted(set(int(x) for x in edges))
        V = sorted(set(x for e in sel for x in E[e]))
    pos = {x: i for i, x in enumerate(V)}
    return V, sel, [pos[E[e][0]] for e in sel], [pos[E[e][1]] for e in sel]


@pytest.mark.parametrize("kind", ["node", "edge"])
def test_subgraph_against_brute_force(kind):
    g = gen.erdos_renyi(60, 0.12, 3, weighted=True)
    R = np.random.default_rng(0).random(g.m) + 0.1
    _, kappa = OE.curvature(g, R)
    pn, pe = OE.sampling_probs(g, kappa, 1e-12)
    if kind == "node":
        idx = S.draw(pn, 25, 9)
        sg = S.node_subgraph(g, idx)
        V, sel, u, v = brute_subgraph(g, nodes=idx)
    else:
        idx = S.draw(pe, 25, 9)
        sg = S.edge_subgraph(g, idx)
        V, sel, u, v = brute_subgraph(g, edges=idx)
    assert sg["nodes"].tolist() == V
    assert sg["edges"].tolist() == sel
    assert sg["u"].tolist() == u and sg["v"].tolist() == v
    assert np.all(sg["u"] < sg["v"])

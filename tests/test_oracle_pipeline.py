"""Pins of the oracle's ERC-LG pipeline (Algorithm 1, Eqs. 3-8).

Each step is checked against something other than itself: the right-hand sides
against the matrix product B^T W^{1/2} Q and a hand-expanded example; the operator
against a dense (L + eps I) X; CG against a dense direct solve; the JL estimate
against bridge edges (exact for every Q), its expectation over seeds and Foster's
theorem; the sampling weights against closed forms.
"""
import math

import numpy as np
import pytest

import gen
from oracle import erc, exact
from oracle import graph as GR
from oracle import hashing as H


# ---- right-hand sides (Section 3.1.2) ------------------------------------------

def test_rhs_hand_expanded_path():
    # path 0-1-2 with weights 4 and 9: edges e0=(0,1), e1=(1,2)
    g = gen.path_graph(3, w=np.array([4.0, 9.0]))
    K, seed = 70, 12
    cols = np.arange(K)
    s = H.signs(seed, K, [0, 1], cols).astype(float)
    expect = np.stack([2 * s[0], -2 * s[0] + 3 * s[1], -3 * s[1]]) / math.sqrt(K)
    Y = erc.rhs(g, K, 0, K, seed)
    assert np.allclose(Y, expect, rtol=0, atol=1e-15)


@pytest.mark.parametrize("col0,ncols", [(0, 32), (5, 70), (64, 64)])
def test_rhs_matches_matrix_product(col0, ncols):
    g = gen.erdos_renyi(60, 0.1, 2, weighted=True)
    K, seed = 160, 4
    Y = erc.rhs(g, K, col0, ncols, seed)
    Yd = exact.dense_rhs(g, K, seed, col0, ncols)
    assert np.allclose(Y, Yd, rtol=0, atol=1e-14)


def test_rhs_columns_sum_to_zero_per_component():
    # unit weights: every entry is an integer times 1/sqrt(K), so sums are exact
    g = gen.from_edges(9, [0, 1, 2, 4, 5, 6], [1, 2, 0, 5, 6, 7])  # node 3 and 8 isolated
    K = 48
    Y = erc.rhs(g, K, 0, K, 3)
    assert np.all(Y[[3, 8]] == 0)
    assert np.all(Y[0:3].sum(axis=0) * math.sqrt(K) == 0)
    assert np.all(np.round(Y[4:8] * math.sqrt(K)).sum(axis=0) == 0)


def test_rhs_f32_is_one_rounding_of_f64():
    g = gen.erdos_renyi(50, 0.1, 6, weighted=True)
    Y64 = erc.rhs(g, 96, 0, 96, 8, "f64")
    Y32 = erc.rhs(g, 96, 0, 96, 8, "f32")
    assert Y32.dtype == np.float32
    assert np.array_equal(Y32, Y64.astype(np.float32))


def test_rhs_row_subset():
    g = gen.erdos_renyi(70, 0.1, 1, weighted=True)
    rows = np.array([5, 0, 69, 33])
    assert np.array_equal(erc.rhs(g, 64, 0, 64, 2, rows=rows), erc.rhs(g, 64, 0, 64, 2)[rows])


# ---- operator and CG (Eq. 5, Section 3.1.3) -------------------------------------

def test_operator_matches_dense():
    g = gen.erdos_renyi(50, 0.15, 3, weighted=True)
    X = np.random.default_rng(0).standard_normal((50, 7))
    L = GR.laplacian(g)
    d = 1e-3
    got = erc.laplacian_apply(L, d, X)
    assert np.allclose(got, (GR.dense_laplacian(g) + d * np.eye(50)) @ X, atol=1e-12)
    assert np.allclose(erc.laplacian_apply(L, d, np.ones((50, 1))), d, atol=1e-12)


def test_cg_matches_direct_solve():
    g = gen.erdos_renyi(120, 0.06, 4, weighted=True)
    L = GR.laplacian(g)
    delta, tol = 1e-3, 1e-10
    Y = erc.rhs(g, 16, 0, 16, 1)
    res = erc.cg_columns(L, delta, Y, tol, 5000)
    Zd = np.linalg.solve(GR.dense_laplacian(g) + delta * np.eye(g.n), Y)
    assert res.converged.all()
    assert np.all(res.relres <= tol)
    assert np.allclose(res.Z, Zd, rtol=0, atol=1e-7 * np.abs(Zd).max())
    true_res = np.linalg.norm(Y - erc.laplacian_apply(L, delta, res.Z), axis=0)
    assert np.all(true_res <= 10 * tol * np.linalg.norm(Y, axis=0))


def test_cg_zero_column_and_iteration_cap():
    g = gen.cycle_graph(40)
    L = GR.laplacian(g)
    Y = np.zeros((40, 3))
    Y[0, 1], Y[20, 1] = 1.0, -1.0
    Y[:, 2] = np.sin(np.arange(40))
    res = erc.cg_columns(L, 1e-6, Y, 1e-12, 3)
    assert res.iters[0] == 0 and res.converged[0] and np.all(res.Z[:, 0] == 0)
    assert res.iters[1] == 3 and not res.converged[1]
    assert res.relres[1] > 1e-12


def test_cg_single_iteration_on_eigenvector():
    # an eigenvector of L + delta I converges in exactly one iteration
    n = 16
    g = gen.cycle_graph(n)
    L = GR.laplacian(g)
    v = np.cos(2 * np.pi * 3 * np.arange(n) / n)[:, None]
    lam = 2 - 2 * np.cos(2 * np.pi * 3 / n)
    res = erc.cg_columns(L, 0.5, v, 1e-10, 10)
    assert res.iters[0] == 1
    assert np.allclose(res.Z[:, 0], v[:, 0] / (lam + 0.5))


# ---- JL estimate (Eqs. 3, 4, 6) -------------------------------------------------

def test_jl_cg_matches_jl_dense():
    g = gen.sbm(3, 40, 0.3, 0.02, 1)
    K, seed, delta = 64, 3, 1e-6
    R, _ = erc.resistance(g, K, 24, delta, 1e-12, 10000, seed)
    Rd = exact.jl_dense_resistance(g, K, seed, delta)
    assert np.allclose(R, Rd, rtol=1e-7)


def test_block_width_does_not_change_result():
    g = gen.erdos_renyi(80, 0.08, 9, weighted=True)
    a, _ = erc.resistance(g, 96, 96, 1e-5, 1e-11, 5000, 2)
    b, _ = erc.resistance(g, 96, 17, 1e-5, 1e-11, 5000, 2)
    assert np.allclose(a, b, rtol=1e-8)
    c1, _ = erc.resistance(g, 96, 32, 1e-5, 1e-11, 5000, 2, col_begin=0, col_end=40)
    c2, _ = erc.resistance(g, 96, 32, 1e-5, 1e-11, 5000, 2, col_begin=40, col_end=96)
    assert np.allclose(a, c1 + c2, rtol=1e-8)


def test_bridges_exact_for_every_projection():
    g = gen.barbell_graph(6, bridge_len=3, seed=4)
    eu, ev, _ = GR.canonical_edges(g)
    w = GR.edge_weights(g)
    bridge = (ev - eu == 1) & (eu >= 5) & (ev <= 8)
    assert bridge.sum() == 3
    for seed in (1, 2, 3):
        R, _ = erc.resistance(g, 8, 8, 1e-10, 1e-13, 10000, seed)
        assert np.allclose(R[bridge], 1.0 / w[bridge], rtol=1e-6)


def test_jl_mean_over_seeds():
    # E_Q[R_hat] = b^T Ld^-1 L Ld^-1 b with Ld = L + delta I, and sd <= R sqrt(2/K)
    g = gen.erdos_renyi(40, 0.15, 2, weighted=True)
    K, delta, S = 32, 1e-3, 60
    L = GR.dense_laplacian(g)
    Li = np.linalg.inv(L + delta * np.eye(g.n))
    M = Li @ L @ Li
    eu, ev, _ = GR.canonical_edges(g)
    expect = M[eu, eu] + M[ev, ev] - 2 * M[eu, ev]
    Lsp = GR.laplacian(g)
    est = np.mean([erc.resistance(g, K, K, delta, 1e-12, 5000, s, L=Lsp)[0]
                   for s in range(S)], axis=0)
    sd = expect * np.sqrt(2.0 / (K * S))
    assert np.all(np.abs(est - expect) < 5 * sd)
    # and the regularised mean is close to the exact resistance
    assert np.allclose(expect, exact.pinv_resistance(g), rtol=1e-2)


def test_foster_statistics_of_estimate():
    # sum_e w_e R_hat_e has mean ~ n - 1 and relative sd <= sqrt(2 / (K (n - 1)))
    g = gen.erdos_renyi(60, 0.1, 3, weighted=True)
    assert GR.components(g) == 1
    K = 512
    R, _ = erc.resistance(g, K, 128, 1e-8, 1e-12, 5000, 21)
    tot = np.sum(GR.edge_weights(g) * R)
    assert abs(tot / (g.n - 1) - 1) < 5 * math.sqrt(2.0 / (K * (g.n - 1)))


def test_jl_error_shrinks_with_k():
    # mean absolute error of R_hat against pinv falls roughly as K^-1/2 (Table 2 trend)
    g = gen.sbm(2, 40, 0.25, 0.03, 5)
    Rx = exact.pinv_resistance(g)
    mae = []
    for K in (64, 256, 1024):
        errs = [np.abs(exact.jl_dense_resistance(g, K, s, 1e-9) - Rx).mean() for s in range(4)]
        mae.append(np.mean(errs))
    assert mae[0] > mae[1] > mae[2]
    ratio = mae[0] / mae[2]  # expected 4 for an exact K^-1/2 law
    assert 2.5 < ratio < 6.5


# ---- sampling weights (Eqs. 7-8, Section 3.2) -----------------------------------

def test_sampling_complete_graph_uniform():
    g = gen.complete_graph(6)
    pn, pe = erc.sampling_probs(g, np.full(g.m, 2.0), 1e-12)
    assert np.allclose(pn, 1 / 6) and np.allclose(pe, 1 / g.m)


def test_sampling_path_closed_form():
    n, eta = 7, 1e-12
    g = gen.path_graph(n)
    kappa = np.array([1.0, 0, 0, 0, 0, 1.0])
    pn, pe = erc.sampling_probs(g, kappa, eta)
    qn = np.array([1, 1, 0, 0, 0, 1, 1]) / (1 + eta)
    assert np.allclose(pn, qn / qn.sum(), rtol=1e-12)
    qe = np.array([2, 1 + math.sqrt(2), 1 + math.sqrt(2), 1 + math.sqrt(2), 1 + math.sqrt(2), 2])
    assert np.allclose(pe, qe / qe.sum(), rtol=1e-12)


def test_sampling_negative_kappa_clamps():
    # star on 6 nodes: every kappa = 4 - 6 = -2 < 0; 2*kmax - kappa = -2 clamps to 0
    g = gen.star_graph(6)
    pn, pe = erc.sampling_probs(g, np.full(5, -2.0), 1e-12)
    assert np.allclose(pe, 0.2)
    assert np.allclose(pn, 1 / 6)


def test_sampling_uniform_fallback_skips_isolated():
    g = gen.from_edges(5, [0, 1], [1, 2])  # nodes 3, 4 isolated
    pn, _ = erc.sampling_probs(g, np.array([0.7, 0.7]), 1e-12)
    assert np.allclose(pn, [1 / 3, 1 / 3, 1 / 3, 0, 0])


def test_sampling_hand_example():
    # triangle 0-1-2 plus pendant 2-3; edges (0,1),(0,2),(1,2),(2,3)
    g = gen.from_edges(4, [0, 0, 1, 2], [1, 2, 2, 3])
    kappa = np.array([3.0, 1.0, 2.0, -1.0])
    eta = 0.5
    den = 3.0 - (-1.0) + eta
    s = (kappa + 1.0) / den
    qn = np.array([s[0] + s[1], s[0] + s[2], s[1] + s[2] + s[3], s[3]])
    pn, pe = erc.sampling_probs(g, kappa, eta)
    assert np.allclose(pn, qn / qn.sum(), rtol=1e-14)
    qe = np.sqrt(np.maximum(6.0 - kappa, 0)) + 1
    assert np.allclose(pe, qe / qe.sum(), rtol=1e-14)


def test_run_end_to_end_small():
    g = gen.make_graph("er2k", use_cache=False)
    res = erc.run(g, gen.CONFIGS["er2k"].params)
    assert all(c.all() for c in res.info.converged)
    assert np.all(res.R > 0)
    assert np.isclose(res.node_prob.sum(), 1) and np.isclose(res.edge_prob.sum(), 1)
    # Foster on the estimate, within the JL spread at K = 32 (sd ~ sqrt(2/(32*1999)))
    assert abs(res.R.sum() / (g.n - 1) - 1) < 5 * math.sqrt(2 / (32 * 1999))

"""Pins of the oracle's Jacobi-preconditioned CG variant (not used by the paper; an
option of the GPU path): the dense direct solve, bit-for-bit equality with plain CG
when the Jacobi scaling is a power of two (a regular graph with delta chosen so that
L_ii + delta = 2^k: every PCG quantity is then an exact rescaling of the CG one, so
using r where s belongs, or r.r where r.s belongs, breaks the equality), the true
residual at the stop, and the iteration saving on a power-law graph (which a scaling
by the diagonal instead of its inverse loses)."""
import numpy as np
import pytest

import gen
from oracle import erc as OE
from oracle import graph as OG


def _dense_solution(g, delta, Y):
    A = OG.dense_laplacian(g) + delta * np.eye(g.n)
    return np.linalg.solve(A, Y)


@pytest.mark.parametrize("weighted", [False, True])
def test_pcg_matches_dense_solve(weighted):
    g = gen.erdos_renyi(300, 0.03, 7, weighted=weighted)
    L = OG.laplacian(g)
    Y = OE.rhs(g, 16, 0, 16, 5, "f64")
    res = OE.pcg_columns(L, 1e-5, Y, 1e-13, 5000)
    assert res.converged.all()
    X = _dense_solution(g, 1e-5, Y)
    assert np.max(np.abs(res.Z - X)) <= 1e-9 * np.max(np.abs(X))


@pytest.mark.parametrize("g,delta", [(gen.cycle_graph(50), 2.0), (gen.complete_graph(9), 8.0)])
def test_pcg_equals_cg_bitwise_when_scaling_is_a_power_of_two(g, delta):
    L = OG.laplacian(g)
    assert np.all(OE.jacobi_inverse(L, delta) == OE.jacobi_inverse(L, delta)[0])
    Y = np.random.default_rng(1).standard_normal((g.n, 6))
    Y -= Y.mean(axis=0)
    a = OE.cg_columns(L, delta, Y, 1e-10, 200)
    b = OE.pcg_columns(L, delta, Y, 1e-10, 200)
    np.testing.assert_array_equal(a.iters, b.iters)
    assert np.array_equal(a.Z, b.Z)


def test_pcg_true_residual_at_stop():
    g = gen.chung_lu(3000, 2.2, 20.0, 20000, seed=3, weighted=True)
    L = OG.laplacian(g)
    Y = OE.rhs(g, 8, 0, 8, 9, "f64")
    tol = 1e-6
    res = OE.pcg_columns(L, 1e-4, Y, tol, 5000)
    assert res.converged.all()
    true_r = Y - OE.laplacian_apply(L, 1e-4, res.Z)
    rel = np.linalg.norm(true_r, axis=0) / np.linalg.norm(Y, axis=0)
    assert np.all(rel <= tol * 1.01)


def test_pcg_needs_far_fewer_iterations_on_power_law_degrees():
    g = gen.chung_lu(20000, 2.3, 40.0, 150000, seed=4, weighted=True)
    L = OG.laplacian(g)
    Y = OE.rhs(g, 4, 0, 4, 2, "f64")
    plain = OE.cg_columns(L, 1e-4, Y, 1e-5, 20000)
    pre = OE.pcg_columns(L, 1e-4, Y, 1e-5, 20000)
    assert plain.converged.all() and pre.converged.all()
    assert pre.iters.max() * 4 < plain.iters.min()

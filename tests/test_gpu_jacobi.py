"""GPU parity of the Jacobi-preconditioned CG variant (ERC_JACOBI) against the oracle's
preconditioned CG (oracle.erc.pcg_columns), at the same tolerances as the plain path,
plus the exact case: when every L_ii + delta is the same power of two the variant is
an exact rescaling of plain CG on the GPU as well, so both give the same bits."""
import numpy as np
import pytest

import gen
from oracle import erc as OE
from oracle import graph as OG

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_27209_amd as E
    return E


def _scaled(g, R_or, k_or, R, k):
    eu, ev, eid = OG.canonical_edges(g)
    rows = OG.entry_rows(g)
    w = np.ones(g.nnz) if g.w is None else np.asarray(g.w, np.float64)
    s = 0.5 * np.bincount(rows, weights=w * R_or[eid], minlength=g.n)
    ks = 2.0 * (s[eu] + s[ev]) / R_or + np.abs(k_or)
    return np.max(np.abs(R - R_or) / R_or), np.max(np.abs(k - k_or) / ks)


@pytest.mark.parametrize("name,rtol", [("er2k", 1e-9), ("sbm20k", 1e-4)])
def test_jacobi_pipeline_parity(name, rtol):
    E = _gpu()
    p = gen.CONFIGS[name].params
    g = gen.make_graph(name)
    R_or, _ = OE.resistance(g, p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed, p.dtype,
                            precond="jacobi")
    _, k_or = OE.curvature(g, R_or)
    G = E.Graph(g.rowptr, g.col, g.w, p.dtype)
    R, info = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed, precond="jacobi")
    _, k = G.curvature(R)
    assert info["cols_unconverged"] == 0 and info["breakdowns"] == 0
    assert info["max_final_relres"] <= p.tol
    rel_R, err_k = _scaled(g, R_or, k_or, R.cpu().numpy(), k.cpu().numpy())
    print(f"{name} jacobi: R {rel_R:.3e} kappa {err_k:.3e} iters {info['iters_max']}")
    assert rel_R <= rtol and err_k <= rtol


def test_jacobi_solve_block_matches_oracle_iterations_fp64():
    E = _gpu()
    p = gen.CONFIGS["er2k"].params
    g = gen.make_graph("er2k")
    G = E.Graph(g.rowptr, g.col, g.w, "f64")
    Z, iters, st = G.debug_solve_block(p.K, p.k_block, p.delta, p.tol, p.seed, 0, p.K,
                                       precond="jacobi")
    Y = OE.rhs(g, p.K, 0, p.K, p.seed, "f64")
    res = OE.pcg_columns(OG.laplacian(g), p.delta, Y, p.tol, p.max_iter)
    assert np.array_equal(np.array(iters), res.iters)
    assert np.allclose(Z.cpu().numpy(), res.Z, rtol=1e-9, atol=1e-9 * np.abs(res.Z).max())


@pytest.mark.parametrize("dtype", ["f32", "f64"])
@pytest.mark.parametrize("g,delta", [(gen.cycle_graph(300), 2.0), (gen.complete_graph(9), 8.0)])
def test_jacobi_equals_plain_when_scaling_is_a_power_of_two(dtype, g, delta):
    E = _gpu()
    G = E.Graph(g.rowptr, g.col, g.w, dtype)
    a, ia = G.resistance(40, 40, delta, 1e-7, 500, 3)
    a = a.clone()
    b, ib = G.resistance(40, 40, delta, 1e-7, 500, 3, precond="jacobi")
    assert ia["iters_total"] == ib["iters_total"]
    assert torch.equal(a, b)


def test_jacobi_cuts_iterations_on_power_law_graph():
    E = _gpu()
    g = gen.make_graph("cl170k")
    p = gen.CONFIGS["cl170k"].params
    G = E.Graph(g.rowptr, g.col, g.w, p.dtype)
    _, plain = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed, col_end=16)
    _, pre = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed, col_end=16,
                          precond="jacobi")
    print(f"cl170k iterations: plain {plain['iters_max']} jacobi {pre['iters_max']}")
    assert pre["iters_max"] * 5 < plain["iters_max"]


def test_unknown_flag_rejected():
    E = _gpu()
    from paper_2609_27209_amd import _abi
    g = gen.make_graph("er2k")
    G = E.Graph(g.rowptr, g.col, g.w, "f64")
    prm = G.params(32, 32, 1e-6, 1e-8, 100, 1)
    prm.flags = 32  # no flag has this bit
    ws = G.workspace(32)
    R = torch.empty(g.m, dtype=torch.float64, device="cuda")
    with pytest.raises(_abi.ErcError) as ei:
        _abi.erc_resistance(G.handle, prm, ws.data_ptr(), ws.numel(), R.data_ptr(),
                            G._stream(), True)
    assert ei.value.status == _abi.ERC_E_INVALID_ARG

"""Replaying captured groups of CG iterations (HIP graphs) gives the same bits as
launching every kernel separately, and fails loudly on non-finite curvature.

Each solve replays its captured group several times per block, with the host's
convergence polls (stream synchronisations) between the replays; repeated solves on
the same handle reuse the cached graph.  Every replayed run is compared bit for bit
with a run that enqueues each launch on its own (ERC_NO_GRAPH), and with the oracle at
the path's tolerance.  The shapes cover fp64 and fp32, unit and weighted graphs, one
and several blocks, and rows split over several blocks of the SpMM (the hub rows of a
Chung-Lu graph, finished by their own launch).
"""
import numpy as np
import pytest

import gen
from oracle import erc as OE

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_27209_amd as E
    return E


CASES = {
    # name: (graph, dtype, K, k_block, delta, tol)
    "er2k_f64": (lambda: gen.make_graph("er2k"), "f64", 32, 32, 1e-6, 1e-8),
    "sbm20k_f32": (lambda: gen.make_graph("sbm20k"), "f32", 64, 64, 1e-5, 1e-6),
    "sbm2k_f32_blocks": (lambda: gen.make_graph("sbm2k"), "f32", 160, 64, 1e-5, 1e-6),
    # 10,000 nodes, one row of 7554 entries split over two SpMM blocks, 394 isolated
    "chung_lu_split_hubs": (lambda: gen.chung_lu(n=10000, gamma=2.0, i0=0.2, m_target=50000,
                                                 seed=18, weighted=True),
                            "f32", 48, 16, 1e-4, 1e-6),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_graph_replay_matches_separate_launches(name):
    E = _gpu()
    make, dtype, K, kb, delta, tol = CASES[name]
    g = make()
    G = E.Graph(g.rowptr, g.col, g.w, solve_dtype=dtype)
    R0, i0 = G.resistance(K, kb, delta, tol, 10000, 17, graph=False)
    ref = R0.cpu().numpy()
    assert i0["cols_unconverged"] == 0 and i0["breakdowns"] == 0
    for rep in range(3):
        R1, i1 = G.resistance(K, kb, delta, tol, 10000, 17)
        torch.cuda.synchronize()
        assert i1["iters_total"] == i0["iters_total"], rep
        np.testing.assert_array_equal(R1.cpu().numpy(), ref)
        # eager work on the same stream between the replayed solves
        _ = G.curvature(R1)
        torch.cuda.synchronize()
    ora, _ = OE.resistance(g, K, kb, delta, tol, 10000, 17, dtype)
    rel = np.max(np.abs(ref - ora) / ora)
    assert rel <= (1e-9 if dtype == "f64" else 1e-4), rel
    print(f"{name}: {i0['iters_max']} iterations, graph replay bit-identical, oracle {rel:.2e}")


def test_split_rows_present_in_hub_case():
    """The hub case really has rows split over several SpMM blocks (checked on the
    host plan through the C ABI's plan check, which also validates the plan)."""
    E = _gpu()
    from paper_2609_27209_amd import _abi
    make = CASES["chung_lu_split_hubs"][0]
    g = make()
    deg = np.diff(np.asarray(g.rowptr))
    assert deg.max() > 4096, "hub case lost its split rows"
    desc, keep = E._desc(g.rowptr, g.col, g.w, "f32")
    _abi.erc_debug_check_plan(desc)
    del keep


@pytest.mark.parametrize("bad", [float("nan"), float("inf"), -float("inf")])
def test_non_finite_curvature_is_reported(bad):
    E = _gpu()
    from paper_2609_27209_amd import _abi
    g = gen.make_graph("er2k")
    G = E.Graph(g.rowptr, g.col, g.w, solve_dtype="f64")
    kappa = torch.linspace(-1.0, 1.0, G.m, dtype=torch.float64, device="cuda")
    kappa[G.m // 3] = bad
    with pytest.raises(_abi.ErcError) as ei:
        G.sampling_probs(kappa, 1e-12)
    assert ei.value.status == _abi.ERC_E_NUMERIC
    # the same call on finite input succeeds afterwards (the flag starts at zero)
    kappa[G.m // 3] = 0.0
    pn, pe = G.sampling_probs(kappa, 1e-12)
    ref_pn, ref_pe = OE.sampling_probs(g, kappa.cpu().numpy(), 1e-12)
    np.testing.assert_allclose(pn.cpu().numpy(), ref_pn, rtol=1e-12, atol=0)
    np.testing.assert_allclose(pe.cpu().numpy(), ref_pe, rtol=1e-12, atol=0)


@pytest.mark.parametrize("name", sorted(CASES))
@pytest.mark.parametrize("precond", ["none", "jacobi"])
def test_early_stop_test_changes_nothing_but_one_spmm(name, precond):
    """The early exact stopping test after each update (ERC_EARLY_STOP; by default only
    on graphs whose SpMM gathers several GB) gives the same bits and iteration counts as
    leaving the test to the next finishing step; it saves at most one SpMM per block,
    the one that would follow the block's last update.  Both with graph replay and with
    separate launches."""
    E = _gpu()
    make, dtype, K, kb, delta, tol = CASES[name]
    g = make()
    G = E.Graph(g.rowptr, g.col, g.w, solve_dtype=dtype)
    for graph in (True, False):
        R0, i0 = G.resistance(K, kb, delta, tol, 10000, 17, graph=graph, precond=precond)
        R0 = R0.cpu().numpy()
        R1, i1 = G.resistance(K, kb, delta, tol, 10000, 17, graph=graph, precond=precond,
                              early_stop=True)
        np.testing.assert_array_equal(R1.cpu().numpy(), R0)
        assert i1["iters_total"] == i0["iters_total"] and i1["iters_max"] == i0["iters_max"]
        assert 0 <= i0["spmm_full"] - i1["spmm_full"] <= i0["blocks"]

"""The entry point that allocates nothing (erc_sampling_probs_static) against the one
that takes a caller scratch buffer (erc_sampling_probs), through the C ABI.

Two calls in a row on one GPU, the second on a smaller graph, so the second call
runs on the fixed scratch array the first one left behind: both must give the same
probabilities, bit for bit, as erc_sampling_probs on the same curvature."""
import numpy as np
import pytest

import gen

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_27209_amd as E
    return E


def _curvature(E, name):
    g = gen.make_graph(name)
    p = gen.CONFIGS[name].params
    G = E.Graph(g.rowptr, g.col, g.w, solve_dtype=p.dtype)
    R, _ = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed)
    _, kappa = G.curvature(R)
    return G, kappa, p.eta


def test_static_scratch_matches_caller_scratch():
    E = _gpu()
    from paper_2609_27209_amd import _abi
    # the larger graph first, then the smaller one on the same array
    for name in ("sbm20k", "er2k"):
        G, kappa, eta = _curvature(E, name)
        ref_pn, ref_pe = G.sampling_probs(kappa, eta)
        pn = torch.full((G.n,), -1.0, dtype=torch.float64, device="cuda")
        pe = torch.full((G.m,), -1.0, dtype=torch.float64, device="cuda")
        stream = torch.cuda.current_stream().cuda_stream
        _abi.erc_sampling_probs_static(G.handle, kappa.data_ptr(), eta, pn.data_ptr(),
                                       pe.data_ptr(), stream)
        torch.cuda.synchronize()
        assert torch.equal(pn, ref_pn), name
        assert torch.equal(pe, ref_pe), name
        assert abs(float(pe.sum()) - 1.0) < 1e-12 and abs(float(pn.sum()) - 1.0) < 1e-12
        print(f"{name}: static-scratch probabilities equal the caller-scratch ones "
              f"({G.n} nodes, {G.m} edges)", flush=True)
        G.close()


def test_static_scratch_non_finite_curvature_gives_nan():
    E = _gpu()
    from paper_2609_27209_amd import _abi
    g = gen.make_graph("er2k")
    G = E.Graph(g.rowptr, g.col, g.w, solve_dtype="f64")
    kappa = torch.linspace(-1.0, 1.0, G.m, dtype=torch.float64, device="cuda")
    kappa[7] = float("nan")
    pn = torch.zeros(G.n, dtype=torch.float64, device="cuda")
    pe = torch.zeros(G.m, dtype=torch.float64, device="cuda")
    _abi.erc_sampling_probs_static(G.handle, kappa.data_ptr(), 1e-12, pn.data_ptr(),
                                   pe.data_ptr(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert torch.isnan(pn).all() and torch.isnan(pe).all()
    # and a finite call afterwards is clean again (every call rewrites the flag)
    kappa[7] = 0.0
    _abi.erc_sampling_probs_static(G.handle, kappa.data_ptr(), 1e-12, pn.data_ptr(),
                                   pe.data_ptr(), torch.cuda.current_stream().cuda_stream)
    ref_pn, ref_pe = G.sampling_probs(kappa, 1e-12)
    torch.cuda.synchronize()
    assert torch.equal(pn, ref_pn) and torch.equal(pe, ref_pe)
    np.testing.assert_allclose(float(pe.sum()), 1.0, rtol=1e-12)

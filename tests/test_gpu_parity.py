"""GPU parity: the HIP path through the C ABI against the CPU oracle on identical seeded
inputs.  Integer work (edge ids, endpoints, projection bits, right-hand sides) must be
bit-exact; floating-point results are compared at 1e-9 (fp64 path) or 1e-4 (fp32
path), relative, with the condition-scaled measures for p and kappa described in the
design notes."""
import math

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


def _graph(E, g, dtype):
    return E.Graph(g.rowptr, g.col, g.w, solve_dtype=dtype)


def _scaled_errors(g, R_or, p_or, k_or, R, p, k):
    """Relative R error; p error over s_u = 1/2 sum w R; kappa error over its first-order
    propagation scale 2 (s_u + s_v)/R + |kappa|."""
    eu, ev, eid = OG.canonical_edges(g)
    rows = OG.entry_rows(g)
    w = np.ones(g.nnz) if g.w is None else np.asarray(g.w, np.float64)
    s = 0.5 * np.bincount(rows, weights=w * R_or[eid], minlength=g.n)
    rel_R = np.max(np.abs(R - R_or) / R_or)
    ps = np.where(s > 0, s, 1.0)
    err_p = np.max(np.abs(p - p_or) / ps)
    ks = 2.0 * (s[eu] + s[ev]) / R_or + np.abs(k_or)
    err_k = np.max(np.abs(k - k_or) / ks)
    return rel_R, err_p, err_k


SMALL = {
    "path5": lambda: gen.path_graph(5),
    "star7_weighted": lambda: gen.star_graph(7, w=np.linspace(0.5, 2.0, 6)),
    "barbell": lambda: gen.barbell_graph(6, bridge_len=3, seed=1),
    "isolated": lambda: gen.from_edges(9, [0, 1, 2, 4, 5], [1, 2, 0, 5, 6]),
    "two_nodes": lambda: gen.from_edges(2, [0], [1]),
    "er300w": lambda: gen.erdos_renyi(300, 0.03, 7, weighted=True),
}


@pytest.mark.parametrize("name", sorted(SMALL))
@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_edge_ids_and_endpoints_bit_exact(name, dtype):
    E = _gpu()
    g = SMALL[name]()
    G = _graph(E, g, dtype)
    eu, ev, eid = OG.canonical_edges(g)
    assert np.array_equal(G.debug_edge_ids().cpu().numpy(), eid)
    u, v = G.edge_endpoints()
    assert np.array_equal(u.cpu().numpy(), eu) and np.array_equal(v.cpu().numpy(), ev)


@pytest.mark.parametrize("dtype,K,col0,ncols", [
    ("f64", 32, 0, 32), ("f64", 200, 64, 40), ("f64", 100, 5, 7), ("f64", 128, 0, 128),
    ("f32", 64, 0, 64), ("f32", 300, 17, 100), ("f32", 256, 128, 128), ("f32", 40, 3, 1),
    ("f32", 512, 0, 256)])
def test_rhs_bit_exact(dtype, K, col0, ncols):
    E = _gpu()
    g = gen.erdos_renyi(400, 0.02, 3, weighted=True)
    G = _graph(E, g, dtype)
    Y = G.debug_rhs(K, col0, ncols, seed=77).cpu().numpy()
    Yo = OE.rhs(g, K, col0, ncols, 77, dtype)
    assert Y.dtype == Yo.dtype
    assert np.array_equal(Y.view(np.uint8), Yo.view(np.uint8))


@pytest.mark.parametrize("dtype,K,col0,ncols", [
    ("f32", 64, 0, 64), ("f32", 96, 40, 40), ("f32", 300, 17, 47), ("f32", 200, 150, 50),
    ("f32", 60, 10, 50), ("f64", 32, 0, 32), ("f64", 100, 60, 8), ("f64", 130, 100, 30),
    ("f32", 512, 128, 128)])
def test_rhs_bit_exact_unit_weights(dtype, K, col0, ncols):
    # unit weights take the integer (ballot) form of the row sums for blocks of up to 64
    # columns, including blocks whose columns straddle two sign words and padded blocks;
    # hub rows span several 64-entry chunks
    E = _gpu()
    g = gen.chung_lu(3000, 2.1, 2.0, 20000, seed=11, weighted=False)
    assert g.w is None and g.degrees().max() > 130
    G = _graph(E, g, dtype)
    Y = G.debug_rhs(K, col0, ncols, seed=31).cpu().numpy()
    Yo = OE.rhs(g, K, col0, ncols, 31, dtype)
    assert Y.dtype == Yo.dtype
    assert np.array_equal(Y.view(np.uint8), Yo.view(np.uint8))


def test_rhs_bit_exact_hub_rows():
    # rows longer than 64 neighbours exercise the 64-wide prefetch windows
    E = _gpu()
    g = gen.chung_lu(3000, 2.1, 2.0, 20000, seed=9, weighted=True)
    assert g.degrees().max() > 300
    G = _graph(E, g, "f32")
    Y = G.debug_rhs(64, 0, 64, seed=5).cpu().numpy()
    assert np.array_equal(Y, OE.rhs(g, 64, 0, 64, 5, "f32"))


@pytest.mark.parametrize("dtype,kb", [("f64", 8), ("f64", 32), ("f64", 128), ("f32", 16),
                                      ("f32", 64), ("f32", 128), ("f32", 256)])
def test_spmm_matches_oracle(dtype, kb):
    E = _gpu()
    g = gen.chung_lu(5000, 2.1, 3.0, 60000, seed=4, weighted=True)  # hub rows -> block tasks
    G = _graph(E, g, dtype)
    rng = np.random.default_rng(1)
    X = rng.standard_normal((g.n, kb)).astype(np.float32 if dtype == "f32" else np.float64)
    delta = 1e-3
    Yg = G.debug_spmm(delta, torch.from_numpy(X)).cpu().numpy().astype(np.float64)
    Yo = OE.laplacian_apply(OG.laplacian(g), delta, X.astype(np.float64))
    # error scale: sum_j w_ij (|x_i| + |x_j|) + delta |x_i|, times the unit roundoff
    L_abs = abs(OG.laplacian(g))
    scale = L_abs @ np.abs(X.astype(np.float64)) + delta * np.abs(X)
    eps = 2.0 ** -24 if dtype == "f32" else 2.0 ** -53
    deg = np.diff(g.rowptr)[:, None] + 2
    assert np.all(np.abs(Yg - Yo) <= 4 * eps * deg * scale + 1e-300)


def test_spmm_multichunk_rows():
    # a star with a 20k-degree centre is split across several blocks
    E = _gpu()
    n = 20001
    g = gen.star_graph(n, w=np.random.default_rng(2).uniform(0.5, 2, n - 1))
    G = _graph(E, g, "f64")
    X = np.random.default_rng(3).standard_normal((n, 16))
    Yg = G.debug_spmm(0.5, torch.from_numpy(X)).cpu().numpy()
    Yo = OE.laplacian_apply(OG.laplacian(g), 0.5, X)
    assert np.allclose(Yg, Yo, rtol=1e-12, atol=1e-9)


def test_spmm_large_grid():
    # 1.2M rows: more than 32 per wave at 8192 blocks, so the SpMM runs on a larger grid
    E = _gpu()
    n = 1_200_001
    g = gen.path_graph(n, w=np.random.default_rng(5).uniform(0.5, 2.0, n - 1))
    G = _graph(E, g, "f32")
    X = np.random.default_rng(6).standard_normal((n, 16)).astype(np.float32)
    Yg = G.debug_spmm(1e-3, torch.from_numpy(X)).cpu().numpy().astype(np.float64)
    L = OG.laplacian(g)
    Yo = OE.laplacian_apply(L, 1e-3, X.astype(np.float64))
    scale = abs(L) @ np.abs(X.astype(np.float64)) + 1e-3 * np.abs(X)
    assert np.all(np.abs(Yg - Yo) <= 4 * 2.0 ** -24 * 4 * scale + 1e-300)


def _run_gpu(E, g, p):
    G = _graph(E, g, p.dtype)
    R, info = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed)
    pp, kk = G.curvature(R)
    pn, pe = G.sampling_probs(kk, p.eta)
    torch.cuda.synchronize()
    return G, R.cpu().numpy(), pp.cpu().numpy(), kk.cpu().numpy(), pn.cpu().numpy(), pe.cpu().numpy(), info


@pytest.mark.parametrize("name,rtol", [("er2k", 1e-9), ("sbm20k", 1e-4)])
def test_pipeline_parity(name, rtol, parity_log):
    E = _gpu()
    wl = gen.CONFIGS[name]
    g = gen.make_graph(name)
    p = wl.params
    ref = OE.run(g, p)
    G, R, pp, kk, pn, pe, info = _run_gpu(E, g, p)
    assert info["cols_unconverged"] == 0 and info["breakdowns"] == 0
    parity_log(name, R=(R, ref.R), p=(pp, ref.p), kappa=(kk, ref.kappa),
               node_prob=(pn, ref.node_prob), edge_prob=(pe, ref.edge_prob))
    rel_R, err_p, err_k = _scaled_errors(g, ref.R, ref.p, ref.kappa, R, pp, kk)
    print(f"{name}: R {rel_R:.3e} p {err_p:.3e} kappa {err_k:.3e} iters {info['iters_max']}")
    assert rel_R <= rtol
    assert err_p <= rtol
    assert err_k <= rtol
    # sampling end to end: total variation distance
    assert 0.5 * np.abs(pn - ref.node_prob).sum() <= rtol
    assert 0.5 * np.abs(pe - ref.edge_prob).sum() <= rtol


@pytest.mark.parametrize("name", ["er2k", "sbm20k"])
def test_sampling_kernels_fed_oracle_kappa(name):
    E = _gpu()
    g = gen.make_graph(name)
    p = gen.CONFIGS[name].params
    ref = OE.run(g, p)
    G = _graph(E, g, p.dtype)
    pn, pe = G.sampling_probs(torch.from_numpy(ref.kappa).cuda(), p.eta)
    assert np.allclose(pn.cpu().numpy(), ref.node_prob, rtol=1e-12, atol=1e-300)
    assert np.allclose(pe.cpu().numpy(), ref.edge_prob, rtol=1e-12, atol=1e-300)


@pytest.mark.parametrize("name", ["er2k", "sbm20k"])
def test_curvature_kernels_fed_oracle_R(name):
    E = _gpu()
    g = gen.make_graph(name)
    p = gen.CONFIGS[name].params
    ref = OE.run(g, p)
    G = _graph(E, g, p.dtype)
    pp, kk = G.curvature(torch.from_numpy(ref.R).cuda())
    po, ko = OE.curvature(g, ref.R)
    w_is_exact = p.dtype == "f64" or g.w is None or g.w.dtype == np.float32
    assert w_is_exact
    assert np.allclose(pp.cpu().numpy(), po, rtol=1e-12, atol=1e-12)
    assert np.allclose(kk.cpu().numpy(), ko, rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("name", sorted(SMALL))
def test_small_graph_pipeline_f64(name):
    E = _gpu()
    g = SMALL[name]()
    K, kb, delta, tol = 48, 16, 1e-8, 1e-12  # three blocks, last one full; ragged padding
    R_or, _ = OE.resistance(g, K, kb, delta, tol, 10000, 5, "f64")
    G = _graph(E, g, "f64")
    R, info = G.resistance(K, kb, delta, tol, 10000, 5)
    R = R.cpu().numpy()
    assert np.allclose(R, R_or, rtol=1e-9)
    p, k = G.curvature(torch.from_numpy(R).cuda())
    po, ko = OE.curvature(g, R)
    assert np.allclose(p.cpu().numpy(), po, rtol=1e-12, atol=1e-12)


def test_ragged_blocks_and_column_ranges():
    E = _gpu()
    g = gen.erdos_renyi(500, 0.02, 11, weighted=True)
    K, delta, tol = 70, 1e-6, 1e-10
    R_or, _ = OE.resistance(g, K, 32, delta, tol, 10000, 3, "f64")
    G = _graph(E, g, "f64")
    R, info = G.resistance(K, 32, delta, tol, 10000, 3)
    assert info["blocks"] == 3
    assert np.allclose(R.cpu().numpy(), R_or, rtol=1e-9)
    # the same sketch in two column ranges, accumulated
    R2, _ = G.resistance(K, 32, delta, tol, 10000, 3, col_begin=0, col_end=30)
    R2 = R2.clone()
    G.resistance(K, 32, delta, tol, 10000, 3, col_begin=30, col_end=70, out=R2, accumulate=True)
    assert np.allclose(R2.cpu().numpy(), R_or, rtol=1e-9)


def test_determinism_bit_identical():
    E = _gpu()
    g = gen.make_graph("sbm20k")
    p = gen.CONFIGS["sbm20k"].params
    G = _graph(E, g, p.dtype)
    a, _ = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed, check_every=3)
    a = a.clone()
    b, _ = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed, check_every=29)
    assert torch.equal(a, b)


def test_not_converged_status():
    E = _gpu()
    g = gen.make_graph("er2k")
    G = _graph(E, g, "f64")
    with pytest.raises(E.ErcNotConverged) as ei:
        G.resistance(32, 32, 1e-6, 1e-8, 1, 101)
    assert ei.value.info.cols_unconverged == 32
    R, info = G.resistance(32, 32, 1e-6, 1e-8, 3, 101, raise_not_converged=False)
    assert info["iters_max"] == 3


def test_solve_block_matches_oracle_cg():
    E = _gpu()
    g = gen.make_graph("er2k")
    p = gen.CONFIGS["er2k"].params
    G = _graph(E, g, "f64")
    Z, iters, st = G.debug_solve_block(p.K, p.k_block, p.delta, p.tol, p.seed, 0, p.K)
    Y = OE.rhs(g, p.K, 0, p.K, p.seed, "f64")
    res = OE.cg_columns(OG.laplacian(g), p.delta, Y, p.tol, p.max_iter)
    assert np.array_equal(np.array(iters), res.iters)
    Zg = Z.cpu().numpy()
    assert np.allclose(Zg, res.Z, rtol=1e-9, atol=1e-9 * np.abs(res.Z).max())


def test_large_grid_solve_matches_oracle_and_repeats():
    # 1.2M rows (the larger SpMM grid): one column of RHS + fp64 CG against the oracle
    # (same iteration count, Z to 1e-9), and two runs bit-identical
    E = _gpu()
    n = 1_200_001
    g = gen.path_graph(n, w=np.random.default_rng(5).uniform(0.5, 2.0, n - 1))
    G = _graph(E, g, "f64")
    K, delta, tol, seed = 16, 1.0, 1e-10, 9
    Z1, it1, _ = G.debug_solve_block(K, 8, delta, tol, seed, 0, 1)
    Z2, it2, _ = G.debug_solve_block(K, 8, delta, tol, seed, 0, 1)
    Z1 = Z1.cpu().numpy()
    assert np.array_equal(Z1, Z2.cpu().numpy()) and list(it1) == list(it2)
    Y = OE.rhs(g, K, 0, 1, seed, "f64")
    res = OE.cg_columns(OG.laplacian(g), delta, Y, tol, 1000)
    assert np.array_equal(np.array(it1), res.iters)
    assert np.allclose(Z1, res.Z, rtol=1e-9, atol=1e-9 * np.abs(res.Z).max())


def test_invalid_arguments_raise():
    E = _gpu()
    g = gen.make_graph("er2k")
    G = _graph(E, g, "f64")
    with pytest.raises(E.ErcError):
        G.resistance(32, 200, 1e-6, 1e-8, 100, 1)      # k_block too wide for fp64
    with pytest.raises(E.ErcError):
        G.resistance(32, 32, -1.0, 1e-8, 100, 1)       # delta <= 0
    with pytest.raises(E.ErcError):
        G.resistance(32, 32, 1e-6, 1e-8, 100, 1, col_begin=10, col_end=5)


def test_solve_info_byte_model():
    # the documented algorithmic byte model of erc_solve_info.bytes_model
    E = _gpu()
    g = gen.make_graph("sbm20k")
    p = gen.CONFIGS["sbm20k"].params
    G = _graph(E, g, p.dtype)
    R, info = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed)
    s, kb, n, nnz, m = 4, 64, g.n, g.nnz, g.m
    spmm = (4 + s) * nnz + 8 * (n + 1) + 3 * s * n * kb
    upd = 7 * s * n * kb
    rhs = (8 + s) * nnz + 3 * s * n * kb
    ed = 2 * nnz + s * n * kb + 16 * m
    want = info["spmm_full"] * (spmm + upd) + info["blocks"] * (rhs + ed)
    assert info["spmm_full"] >= info["iters_max"]
    assert info["bytes_model"] == pytest.approx(want, rel=1e-12)

"""Parity over a sweep of seeded graph shapes: power-law graphs whose rows reach every
SpMM work path (rows gathered by a lane group, chunks gathered by the whole wavefront,
block tasks above 1024 entries, hub rows above 4096 entries split over several blocks),
with isolated nodes and many components, weighted and unit, in both working
precisions.  Every case checks the operator (L + delta I) X against the oracle within
its rounding bound, and the whole path (resistance, curvature, sampling
probabilities) against the oracle at 1e-9 (fp64) or 1e-4 (fp32), with ragged column
blocks.  The host plan check on the same shapes needs no GPU."""
import numpy as np
import pytest

import gen
from gen.configs import SolveParams
from oracle import erc as OE
from oracle import graph as OG

torch = pytest.importorskip("torch")

# name -> Chung-Lu arguments; realised: cl10000: 6 rows > 1024 (block tasks), one of
# 7554 entries > 4096 (split over two blocks), 394 isolated; cl3000: 7 rows > 256 (long
# wavefront rows), 177 isolated, 180 components; cl4097: largest component only (4066
# nodes), 11 rows > 256; cl1500: unit weights, 40 rows > 32; cl777: every row <= 32;
# cl65: one dense component, every row between 12 and 54 entries
SHAPES = {
    "cl10000_g20": dict(n=10000, gamma=2.0, i0=0.2, m_target=50000, seed=18, weighted=True),
    "cl3000_g21": dict(n=3000, gamma=2.1, i0=1.0, m_target=12000, seed=11, weighted=True),
    "cl4097_g23_lcc": dict(n=4097, gamma=2.3, i0=2.0, m_target=24000, seed=13, weighted=True,
                           keep_largest=True),
    "cl1500_g25_unit": dict(n=1500, gamma=2.5, i0=3.0, m_target=6000, seed=12),
    "cl777_g30": dict(n=777, gamma=3.0, i0=10.0, m_target=2000, seed=14, weighted=True),
    "cl65_dense": dict(n=65, gamma=2.2, i0=1.0, m_target=900, seed=15, weighted=True),
}

_CACHE = {}


def _shape(name):
    if name not in _CACHE:
        _CACHE[name] = gen.graphs.chung_lu(**SHAPES[name])
    return _CACHE[name]


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_27209_amd as E
    return E


def test_sweep_shapes_reach_every_work_path():
    deg = {k: np.diff(_shape(k).rowptr) for k in SHAPES}
    assert (deg["cl10000_g20"] > 4096).sum() >= 1
    assert (deg["cl10000_g20"] > 1024).sum() >= 5
    assert (deg["cl3000_g21"] > 256).sum() >= 5
    assert any((d == 0).sum() > 100 for d in deg.values())
    assert any(((d > 32) & (d <= 256)).sum() > 10 for d in deg.values())
    assert deg["cl777_g30"].max() <= 32


@pytest.mark.parametrize("name", sorted(SHAPES))
def test_sweep_host_plan(name):
    import paper_2609_27209_amd as E
    from paper_2609_27209_amd import _abi

    g = _shape(name)
    for dt in ("f32", "f64"):
        d, keep = E._desc(g.rowptr, g.col, g.w, dt)
        _abi.erc_debug_check_plan(d)


@pytest.mark.gpu
@pytest.mark.parametrize("name", sorted(SHAPES))
@pytest.mark.parametrize("dtype,kb", [("f64", 8), ("f64", 64), ("f32", 16), ("f32", 128)])
def test_sweep_spmm(name, dtype, kb):
    E = _gpu()
    g = _shape(name)
    G = E.Graph(g.rowptr, g.col, g.w, solve_dtype=dtype)
    rng = np.random.default_rng(kb + g.n)
    X = rng.standard_normal((g.n, kb)).astype(np.float32 if dtype == "f32" else np.float64)
    delta = 1e-3
    Yg = G.debug_spmm(delta, torch.from_numpy(X)).cpu().numpy().astype(np.float64)
    L = OG.laplacian(g)
    Yo = OE.laplacian_apply(L, delta, X.astype(np.float64))
    # each output is a sum of deg + 1 terms in the working precision
    scale = abs(L) @ np.abs(X.astype(np.float64)) + delta * np.abs(X)
    eps = 2.0 ** -24 if dtype == "f32" else 2.0 ** -53
    deg = np.diff(g.rowptr)[:, None] + 2
    assert np.all(np.abs(Yg - Yo) <= 4 * eps * deg * scale + 1e-300)


def _scaled(g, ref, R, p, k):
    eu, ev, eid = OG.canonical_edges(g)
    rows = OG.entry_rows(g)
    w = np.ones(g.nnz) if g.w is None else np.asarray(g.w, np.float64)
    s = 0.5 * np.bincount(rows, weights=w * ref.R[eid], minlength=g.n)
    rel_R = np.max(np.abs(R - ref.R) / ref.R)
    err_p = np.max(np.abs(p - ref.p) / np.where(s > 0, s, 1.0))
    err_k = np.max(np.abs(k - ref.kappa) / (2.0 * (s[eu] + s[ev]) / ref.R + np.abs(ref.kappa)))
    return rel_R, err_p, err_k


@pytest.mark.gpu
@pytest.mark.parametrize("name", sorted(SHAPES))
@pytest.mark.parametrize("dtype", ["f64", "f32"])
def test_sweep_pipeline(name, dtype):
    E = _gpu()
    g = _shape(name)
    # 40 columns in blocks of 16: two full blocks and a ragged one of 8
    if dtype == "f64":
        p = SolveParams(K=40, k_block=16, delta=1e-4, tol=1e-10, dtype="f64", seed=31)
        rtol = 1e-9
    else:
        p = SolveParams(K=40, k_block=16, delta=1e-4, tol=1e-6, dtype="f32", seed=31)
        rtol = 1e-4
    ref = OE.run(g, p)
    G = E.Graph(g.rowptr, g.col, g.w, solve_dtype=dtype)
    R, info = G.resistance(p.K, p.k_block, p.delta, p.tol, p.max_iter, p.seed)
    pp, kk = G.curvature(R)
    pn, pe = G.sampling_probs(kk, p.eta)
    torch.cuda.synchronize()
    assert info["blocks"] == 3 and info["cols_unconverged"] == 0 and info["breakdowns"] == 0
    rel_R, err_p, err_k = _scaled(g, ref, R.cpu().numpy(), pp.cpu().numpy(), kk.cpu().numpy())
    print(f"{name} {dtype}: R {rel_R:.2e} p {err_p:.2e} kappa {err_k:.2e} "
          f"iters {info['iters_max']} (oracle {max(int(np.max(i)) for i in ref.info.iters)})")
    assert rel_R <= rtol
    assert err_p <= rtol
    assert err_k <= rtol
    assert 0.5 * np.abs(pn.cpu().numpy() - ref.node_prob).sum() <= rtol
    assert 0.5 * np.abs(pe.cpu().numpy() - ref.edge_prob).sum() <= rtol

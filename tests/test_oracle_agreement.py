"""Pins of the agreement metrics and of the oracle side of the curvature-agreement
study (Section 4, Table 2): closed-form rank cases, an independent library
implementation of Spearman's rho, the delta -> 0 limit of the regularised resistance
and the K^(-1/2) error decay of the JL estimate."""
import json
import os

import numpy as np
import pytest
from scipy import stats

import gen
from oracle import agreement as AG
from oracle import erc as OE
from oracle import exact as EX

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "sbm2k_agreement.npz")


def test_mae_and_sign_by_hand():
    assert AG.mae([1.0, -2.0, 3.0], [1.5, -2.0, 2.0]) == pytest.approx(0.5)
    assert AG.sign_agreement([1.0, -1.0, 0.0, 2.0], [3.0, -2.0, 0.0, -1.0]) == 0.75
    # zero is its own sign class: 0 against a negative (or a positive) disagrees
    assert AG.sign_agreement([0.0, 2.0, -1.0], [-3.0, 1.0, 0.0]) == pytest.approx(1 / 3)


def test_average_ranks_ties():
    np.testing.assert_array_equal(AG.average_ranks([10, 20, 20, 5]), [2.0, 3.5, 3.5, 1.0])
    np.testing.assert_array_equal(AG.average_ranks([7, 7, 7]), [2.0, 2.0, 2.0])


def test_spearman_closed_forms():
    a = np.arange(1.0, 6.0)
    # no ties: rho = 1 - 6 sum d^2 / (n (n^2 - 1)); ranks of b are 2 1 4 3 5, sum d^2 = 4
    assert AG.spearman(a, [6.0, 5.0, 8.0, 7.0, 9.0]) == pytest.approx(1 - 6 * 4 / (5 * 24))
    x = np.random.default_rng(0).normal(size=200)
    assert AG.spearman(x, np.exp(x)) == pytest.approx(1.0)
    assert AG.spearman(x, -x ** 3) == pytest.approx(-1.0)


def test_spearman_matches_scipy_with_ties():
    rng = np.random.default_rng(1)
    a = rng.integers(0, 20, size=500).astype(float)
    b = a + rng.integers(0, 5, size=500)
    assert AG.spearman(a, b) == pytest.approx(stats.spearmanr(a, b).statistic, abs=1e-12)


def small_sbm():
    return gen.sbm(4, 75, 8.0 / 74.0, 1.0 / 225.0, 9)


def test_regularised_resistance_tends_to_pinv():
    g = small_sbm()
    _, kp = OE.curvature(g, EX.pinv_resistance(g))
    errs = []
    for eps in (1e-3, 1e-4, 1e-5):
        _, kr = OE.curvature(g, EX.reg_resistance(g, eps))
        errs.append(AG.mae(kr, kp))
    # the bias of b^T (L + eps I)^-1 b is first order in eps
    assert errs[1] / errs[0] == pytest.approx(0.1, rel=0.05)
    assert errs[2] / errs[1] == pytest.approx(0.1, rel=0.05)
    assert AG.sign_agreement(kr, kp) == 1.0


def test_jl_error_decays_as_inverse_sqrt_k():
    g = small_sbm()
    _, kp = OE.curvature(g, EX.pinv_resistance(g))
    m = {}
    for K in (64, 1024):
        _, kj = OE.curvature(g, EX.jl_dense_resistance(g, K, 11, 1e-6))
        m[K] = AG.metrics(kj, kp)
    assert 3.0 < m[64]["mae"] / m[1024]["mae"] < 5.5   # sqrt(16) = 4
    assert m[1024]["spearman"] > m[64]["spearman"]
    assert m[1024]["sign"] > m[64]["sign"]


@pytest.mark.skipif(not os.path.exists(GOLDEN), reason="agreement goldens not written")
def test_stored_agreement_goldens_consistent():
    with np.load(GOLDEN) as f:
        meta = json.loads(str(f["meta"]))
        kp = f["kappa_pinv"]
        assert AG.mae(f["kappa_reg"], kp) < 1e-4
        maes = []
        for K in meta["Ks"]:
            mk = AG.metrics(f[f"kappa_jl_{K}"], kp)
            assert mk == pytest.approx(meta["oracle_metrics"][f"JL{K}"])
            maes.append(mk["mae"])
    assert maes[0] > maes[1] > maes[2]
    assert 1.6 < maes[0] / maes[2] < 2.5

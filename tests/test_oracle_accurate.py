"""Pins of the oracle's twice-working-precision inner products against exact rational
arithmetic (Ogita, Rump & Oishi 2005 bound: |dot2 - x.y| <= eps |x.y| + gamma_n^2 sum |x_i y_i|)."""
from fractions import Fraction

import numpy as np
import pytest

from oracle.accurate import dot2_columns, two_prod, two_sum

EPS = 2.0 ** -53


def exact_dot(x, y):
    return sum((Fraction(float(a)) * Fraction(float(b)) for a, b in zip(x, y)), Fraction(0))


def ill_conditioned(n, cond_exp, rng):
    # half the terms large with random signs, then a correction that cancels them
    x = rng.standard_normal(n) * 2.0 ** rng.integers(0, cond_exp, n)
    y = rng.standard_normal(n)
    # make the sum nearly cancel: adjust the last entry exactly in rationals
    s = exact_dot(x[:-1], y[:-1])
    x[-1] = float(-s / Fraction(float(y[-1])))
    return x, y


def test_error_free_transformations():
    rng = np.random.default_rng(0)
    a = rng.standard_normal(1000) * 1e3
    b = rng.standard_normal(1000) * 1e-3
    s, e = two_sum(a, b)
    p, f = two_prod(a, b)
    for k in range(0, 1000, 37):
        assert Fraction(float(s[k])) + Fraction(float(e[k])) == Fraction(float(a[k])) + Fraction(float(b[k]))
        assert Fraction(float(p[k])) + Fraction(float(f[k])) == Fraction(float(a[k])) * Fraction(float(b[k]))


@pytest.mark.parametrize("n,cond", [(10, 10), (300, 30), (2000, 50)])
def test_dot2_within_published_bound(n, cond):
    rng = np.random.default_rng(n)
    cols = [ill_conditioned(n, cond, rng) for _ in range(4)]
    X = np.stack([c[0] for c in cols], axis=1)
    Y = np.stack([c[1] for c in cols], axis=1)
    got = dot2_columns(X, Y)
    gamma = n * EPS / (1 - n * EPS)
    for c in range(4):
        ex = exact_dot(X[:, c], Y[:, c])
        absum = float(sum(abs(Fraction(float(a)) * Fraction(float(b))) for a, b in zip(X[:, c], Y[:, c])))
        err = abs(Fraction(float(got[c])) - ex)
        assert float(err) <= EPS * abs(float(ex)) + gamma ** 2 * absum


def test_dot2_beats_plain_sum_on_cancellation():
    rng = np.random.default_rng(7)
    x, y = ill_conditioned(500, 40, rng)
    ex = float(exact_dot(x, y))
    plain = float(np.dot(x, y))
    acc = float(dot2_columns(x[:, None], y[:, None])[0])
    assert abs(acc - ex) <= abs(plain - ex)
    assert abs(acc - ex) <= 1e-20 * np.sum(np.abs(x * y)) + EPS * abs(ex)


def test_dot2_shapes():
    X = np.arange(12.0).reshape(4, 3)
    assert np.array_equal(dot2_columns(X, X), (X * X).sum(axis=0))
    assert dot2_columns(np.zeros((0, 2)), np.zeros((0, 2))).shape == (2,)
    assert dot2_columns(np.ones((1, 2)), np.full((1, 2), 3.0)).tolist() == [3.0, 3.0]

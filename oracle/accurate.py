"""Inner products in twice the working precision (oracle side).

The conjugate-gradient recurrences of Section 3.1.3 are driven by inner products
(p.q for the step, r.r for the direction update and the stopping test).  Summation
error in those products is the largest rounding effect in an fp64 CG: on the 2000-node
workload a plain fp64 sum moves R by up to 5e-9 against an extended-precision run,
while the operator and vector updates contribute about 2e-10.  The oracle therefore
evaluates every CG inner product with the Dot2 scheme of Ogita, Rump and Oishi
("Accurate sum and dot product", SIAM J. Sci. Comput. 26(6), 2005): each product is
split exactly into a rounded part and its error (Dekker's TwoProduct with Veltkamp
splitting, no FMA needed), the rounded parts are summed pairwise with Knuth's TwoSum
collecting every rounding error, and the collected errors are added at the end.  The
result is as accurate as if computed in twice the working precision and then rounded.
"""
from __future__ import annotations

import numpy as np

_SPLIT = 134217729.0  # 2^27 + 1: Veltkamp splitting constant for binary64


def two_sum(a, b):
    """s = fl(a + b) and the exact error e with a + b = s + e (Knuth)."""
    s = a + b
    z = s - a
    e = (a - (s - z)) + (b - z)
    return s, e


def two_prod(a, b):
    """p = fl(a * b) and the exact error e with a * b = p + e (Dekker)."""
    p = a * b
    ca = _SPLIT * a
    ah = ca - (ca - a)
    al = a - ah
    cb = _SPLIT * b
    bh = cb - (cb - b)
    bl = b - bh
    e = ((ah * bh - p) + ah * bl + al * bh) + al * bl
    return p, e


def dot2_columns(X: np.ndarray, Y: np.ndarray) -> np.ndarray:
    """Column-wise dot products sum_i X[i, c] * Y[i, c], accurate to about fp64 squared."""
    X = np.asarray(X, dtype=np.float64)
    Y = np.asarray(Y, dtype=np.float64)
    s, e = two_prod(X, Y)
    err = e.sum(axis=0)
    while s.shape[0] > 1:
        if s.shape[0] % 2:
            s = np.concatenate([s, np.zeros((1,) + s.shape[1:])], axis=0)
        s, t = two_sum(s[0::2], s[1::2])
        err = err + t.sum(axis=0)
    if s.shape[0] == 0:
        return np.zeros(X.shape[1:])
    return s[0] + err

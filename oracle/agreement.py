"""Agreement metrics for curvature estimates (test infrastructure, like all of oracle/).

Section 4 (numerical agreement of curvature estimates, Table 2) compares edge
curvatures from an approximate scheme with those from the pseudoinverse-based
resistance curvature by three numbers: the mean absolute error, the Spearman rank
correlation and the sign agreement.  Written from their textbook definitions:

* mae(a, b)            = (1/m) sum_e |a_e - b_e|
* spearman(a, b)       = Pearson correlation of the rank vectors of a and b, where
                         tied values share the mean of the positions they occupy
* sign_agreement(a, b) = (1/m) #{e : sign(a_e) = sign(b_e)}, sign in {-1, 0, +1}
"""
from __future__ import annotations

import numpy as np


def mae(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.mean(np.abs(a - b)))


def average_ranks(x) -> np.ndarray:
    """Ranks 1..m of x; each run of equal values gets the mean rank of the run."""
    x = np.asarray(x, dtype=np.float64)
    order = np.argsort(x, kind="stable")
    xs = x[order]
    ranks = np.empty(x.size, dtype=np.float64)
    i = 0
    while i < x.size:
        j = i
        while j + 1 < x.size and xs[j + 1] == xs[i]:
            j += 1
        ranks[order[i:j + 1]] = 0.5 * (i + j) + 1.0  # mean of positions i+1 .. j+1
        i = j + 1
    return ranks


def pearson(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    da = a - a.mean()
    db = b - b.mean()
    return float(np.sum(da * db) / np.sqrt(np.sum(da * da) * np.sum(db * db)))


def spearman(a, b) -> float:
    return pearson(average_ranks(a), average_ranks(b))


def sign_agreement(a, b) -> float:
    return float(np.mean(np.sign(np.asarray(a, np.float64)) == np.sign(np.asarray(b, np.float64))))


def metrics(estimate, reference) -> dict:
    return {"mae": mae(estimate, reference), "spearman": spearman(estimate, reference),
            "sign": sign_agreement(estimate, reference)}

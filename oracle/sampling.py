"""Curvature-guided subgraph draws (oracle side; test infrastructure like all of oracle/).

Section 3.2 turns the normalised node weights of Eq. 7 and edge weights of Eq. 8 into
sampling distributions; the experiments of Section 4 draw GraphSAINT-style training
subgraphs from them.  The paper fixes neither the random generator nor how a draw is
turned into an index; this oracle reads the draw as follows.

Draw (inverse CDF over exact integers):
* W_i = floor(P_i * 2^62) for every item i (a power-of-two scaling of the fp64
  probability, so exact), T = sum_i W_i, C_i = sum_{j < i} W_j (exact in 64 bits,
  T < 2^63 for probabilities that sum to one up to rounding).
* Draw d takes X = x_hi * 2^64 + x_lo with x_hi, x_lo outputs 2d and 2d+1 of SplitMix64
  started from base(seed) (the same generator as the projection signs, see hashing),
  and the target t = floor(X * T / 2^128), uniform on [0, T) up to 2^-65 relative.
* The drawn item is the i with C_i <= t < C_i + W_i; items with W_i = 0 never appear.

Subgraph (the paper: selected edges and their endpoints form the edge-sampled subgraph;
node sampling follows GraphSAINT's node sampler, read here as the subgraph induced on
the distinct drawn nodes):
* nodes are listed in increasing original id and renumbered 0..n_s-1 in that order;
* edges are listed in increasing canonical id, with their endpoints (u < v) renumbered.
"""
from __future__ import annotations

import numpy as np

from . import graph as GR
from . import hashing as H

SCALE_BITS = 62


def integer_weights(prob) -> np.ndarray:
    """W_i = floor(P_i * 2^62) as uint64."""
    P = np.asarray(prob, dtype=np.float64)
    if not np.all(np.isfinite(P)) or np.any(P < 0) or np.any(P > 1):
        raise ValueError("probabilities must be finite and in [0, 1]")
    # every product is an integer-valued double below 2^63 or below 1, so the floor and
    # the conversion are exact
    return np.floor(np.ldexp(P, SCALE_BITS)).astype(np.uint64)


def draw_targets(seed: int, T: int, draws: int) -> list:
    """t_d = floor((x_hi 2^64 + x_lo) T / 2^128) for d = 0 .. draws-1, Python ints."""
    words = H.splitmix64(int(H.base(seed)), 2 * draws)
    out = []
    for d in range(draws):
        X = (int(words[2 * d]) << 64) | int(words[2 * d + 1])
        out.append((X * T) >> 128)
    return out


def draw(prob, draws: int, seed: int) -> np.ndarray:
    """Indices of `draws` independent draws from the distribution `prob`."""
    W = integer_weights(prob)
    # probabilities that sum to at most 1.5 keep sum_i W_i below 2^63, so the uint64
    # sums below are exact
    if not float(np.sum(np.asarray(prob, dtype=np.float64))) <= 1.5:
        raise ValueError("probabilities sum above 1.5")
    C = np.zeros(W.size + 1, dtype=np.uint64)
    np.cumsum(W, out=C[1:])
    T = int(C[-1])
    if T == 0:
        raise ValueError("all weights are zero")
    return select(C, draw_targets(seed, T, draws))


def select(C, targets) -> np.ndarray:
    """For each target t in [0, C[-1]), the item i with C[i] <= t < C[i+1], where C holds
    the n+1 exclusive prefix sums of the integer weights (C[0] = 0).  Such an i has
    W_i = C[i+1] - C[i] > 0, so items of weight zero are never selected."""
    C = np.asarray(C, dtype=np.uint64)
    out = np.empty(len(targets), dtype=np.int64)
    for d, t in enumerate(targets):
        # the last i with C_i <= t
        out[d] = int(np.searchsorted(C, np.uint64(t), side="right")) - 1
    return out


def node_subgraph(g, node_idx):
    """Subgraph induced on the distinct drawn nodes."""
    keep = np.zeros(g.n, dtype=bool)
    keep[np.asarray(node_idx, dtype=np.int64)] = True
    eu, ev, _ = GR.canonical_edges(g)
    ekeep = keep[eu] & keep[ev]
    return _relabel(keep, np.nonzero(ekeep)[0], eu, ev)


def edge_subgraph(g, edge_idx):
    """The distinct drawn edges and their endpoints."""
    eu, ev, _ = GR.canonical_edges(g)
    ekeep = np.zeros(g.m, dtype=bool)
    ekeep[np.asarray(edge_idx, dtype=np.int64)] = True
    keep = np.zeros(g.n, dtype=bool)
    keep[eu[ekeep]] = True
    keep[ev[ekeep]] = True
    return _relabel(keep, np.nonzero(ekeep)[0], eu, ev)


def _relabel(keep, edges, eu, ev):
    nodes = np.nonzero(keep)[0]
    new_id = np.full(keep.size, -1, dtype=np.int64)
    new_id[nodes] = np.arange(nodes.size)
    return {"nodes": nodes.astype(np.int64), "edges": edges.astype(np.int64),
            "u": new_id[eu[edges]], "v": new_id[ev[edges]]}

"""Pins of the oracle's projection generator (Section 3.1.2: Q has independent
+-1/sqrt(K) entries; SplitMix64 realises the draw)."""
import os

import numpy as np
import pytest

from oracle import hashing as H


def _vectors(golden_dir):
    out = []
    with open(os.path.join(golden_dir, "splitmix64_vectors.txt")) as f:
        for line in f:
            if line.startswith("state"):
                head, vals = line.split(":")
                out.append((int(head.split()[1]), [int(x) for x in vals.split()]))
    return out


def test_splitmix64_published_vectors(golden_dir):
    vecs = _vectors(golden_dir)
    assert len(vecs) == 2
    for state, expect in vecs:
        got = H.splitmix64(state, len(expect))
        assert [int(x) for x in got] == expect


def test_sign_word_is_stream_output():
    # word(e, i) is output number e*W + i of the generator started at base(seed)
    seed, K = 7, 200
    W = H.words_per_edge(K)
    assert W == 4
    stream = H.splitmix64(int(H.base(seed)), 40)
    for e in range(10):
        for i in range(W):
            assert int(H.sign_words(seed, K, e, i)) == int(stream[e * W + i])


def test_base_is_first_output():
    assert int(H.base(0)) == 16294208416658607535


def test_signs_bit_layout():
    seed, K = 3, 130
    e = np.array([0, 5, 17])
    cols = np.arange(K)
    s = H.signs(seed, K, e, cols)
    for a, ee in enumerate(e):
        for c in cols:
            word = int(H.sign_words(seed, K, ee, c // 64))
            bit = (word >> int(c % 64)) & 1
            assert s[a, c] == (1 - 2 * bit)


def test_sign_statistics():
    # balance and pairwise independence of the +-1 entries, within 5 sigma
    seed, K, m = 11, 256, 4000
    s = H.signs(seed, K, np.arange(m), np.arange(K)).astype(np.float64)
    N = s.size
    assert abs(s.mean()) < 5 / np.sqrt(N)
    # column Gram matrix: E[Q^T Q] = I  (off-diagonal sd 1/sqrt(m))
    G = s.T @ s / m
    off = G[~np.eye(K, dtype=bool)]
    assert np.abs(off).max() < 6 / np.sqrt(m)
    assert abs(off.mean()) < 5 / np.sqrt(m * K * (K - 1))
    # row Gram matrix (edges against edges) for a subset
    Gr = s[:300] @ s[:300].T / K
    offr = Gr[~np.eye(300, dtype=bool)]
    assert np.abs(offr).max() < 6 / np.sqrt(K)
    # neighbouring edges / columns are not correlated bitwise
    assert abs((s[1:] * s[:-1]).mean()) < 5 / np.sqrt(N)
    assert abs((s[:, 1:] * s[:, :-1]).mean()) < 5 / np.sqrt(N)


def test_seeds_differ():
    a = H.signs(1, 64, np.arange(100), np.arange(64))
    b = H.signs(2, 64, np.arange(100), np.arange(64))
    assert (a != b).mean() > 0.4


@pytest.mark.parametrize("K", [1, 63, 64, 65, 128])
def test_words_per_edge(K):
    assert H.words_per_edge(K) == -(-K // 64)

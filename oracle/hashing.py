"""SplitMix64 and the projection signs (oracle side).

The paper draws Q with independent entries uniform on {+1/sqrt(K), -1/sqrt(K)}
(Section 3.1.2 and the streamed Q of Algorithm 1) but names no generator.  This
oracle realises that draw with a counter-based generator so each entry can be
regenerated on demand:

* SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number
  generators", OOPSLA 2014): state advances by the golden-ratio increment
  0x9E3779B97F4A7C15, and each output is the state passed through the 64-bit
  finaliser (xor-shift 30, multiply 0xBF58476D1CE4E5B9, xor-shift 27, multiply
  0x94D049BB133111EB, xor-shift 31).  Output k of a generator in state s is
  finalise(s + (k+1)*increment), all mod 2^64.
* base(seed) = the first output of SplitMix64 seeded with ``seed``.
* word(e, i) = output number e*W + i of SplitMix64 started from state base(seed),
  with W = ceil(K/64) words per edge.
* sign(e, c) = +1 if bit (c mod 64) of word(e, c // 64) is 0, else -1; the JL
  entry is Q[e, c] = sign(e, c) / sqrt(K), c being the global column index.
"""
from __future__ import annotations

import numpy as np

U64 = np.uint64
GOLDEN = U64(0x9E3779B97F4A7C15)
MUL1 = U64(0xBF58476D1CE4E5B9)
MUL2 = U64(0x94D049BB133111EB)


def finalise(z):
    """SplitMix64 output finaliser on uint64 values (array or scalar), mod 2^64."""
    z = np.asarray(z, dtype=U64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> U64(30))) * MUL1
        z = (z ^ (z >> U64(27))) * MUL2
    return z ^ (z >> U64(31))


def splitmix64(state: int, count: int) -> np.ndarray:
    """The first ``count`` outputs of SplitMix64 started from ``state``."""
    k = np.arange(1, count + 1, dtype=U64)
    with np.errstate(over="ignore"):
        return finalise(U64(state) + k * GOLDEN)


def base(seed: int) -> np.uint64:
    return U64(splitmix64(seed, 1)[0])


def words_per_edge(K: int) -> int:
    return (int(K) + 63) // 64


def sign_words(seed: int, K: int, e, word_index) -> np.ndarray:
    """word(e, i) for broadcastable arrays of edge ids and word indices."""
    W = U64(words_per_edge(K))
    e = np.asarray(e, dtype=U64)
    i = np.asarray(word_index, dtype=U64)
    with np.errstate(over="ignore"):
        counter = e * W + i + U64(1)
        return finalise(base(seed) + counter * GOLDEN)


def signs(seed: int, K: int, e, cols) -> np.ndarray:
    """+-1 (int8) matrix of shape (len(e), len(cols)) for global columns ``cols``.

    Each sign word is generated once per edge and 64-column word, then every column
    reads its bit from it.
    """
    e = np.asarray(e, dtype=np.int64).reshape(-1, 1)
    cols = np.asarray(cols, dtype=np.int64).reshape(-1)
    wi, pick = np.unique(cols // 64, return_inverse=True)
    words = sign_words(seed, K, e, wi.reshape(1, -1))[:, pick]
    bits = (words >> (cols % 64).astype(U64).reshape(1, -1)) & U64(1)
    return (1 - 2 * bits.astype(np.int8)).astype(np.int8)

"""Pins of the oracle's random-number layer against independent references.

- Philox4x64-10 against numpy.random.Philox (numpy's own implementation of the
  same published generator).  numpy increments its 256-bit counter before each
  block of four words, so Philox(c) is numpy's first block for counter c - 1.
- The multiply-shift integer draw against Python big-integer arithmetic.
- The keying of a request's words: word i of (seed, v, m, l) is lane i & 3 of
  Philox at key (seed, 0), counter (i >> 2, v, m, l).
"""
import random

import numpy as np
import pytest

import oracle

M64 = (1 << 64) - 1


def numpy_philox(counter, key):
    c = 0
    for w, x in enumerate(counter):
        c |= int(x) << (64 * w)
    c = (c - 1) % (1 << 256)
    words = [(c >> (64 * w)) & M64 for w in range(4)]
    g = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=np.array(words, dtype=np.uint64))
    return [int(x) for x in g.random_raw(4)]


def test_philox_zero_vector_matches_numpy():
    assert oracle.philox4x64_10([0, 0, 0, 0], [0, 0]) == numpy_philox([0, 0, 0, 0], [0, 0])


@pytest.mark.parametrize("trial", range(200))
def test_philox_random_vectors_match_numpy(trial):
    rng = random.Random(1000 + trial)
    ctr = [rng.getrandbits(64) for _ in range(4)]
    if trial % 4 == 0:
        ctr[0] = 0          # borrow chain through the low words on numpy's side
    if trial % 8 == 0:
        ctr[1] = 0
    key = [rng.getrandbits(64), rng.getrandbits(64)]
    assert oracle.philox4x64_10(ctr, key) == numpy_philox(ctr, key)


def test_philox_small_counters_match_numpy():
    for i in range(64):
        for v in (0, 1, 7, 123456):
            ctr = [i, v, 3, 1]
            assert oracle.philox4x64_10(ctr, [42, 0]) == numpy_philox(ctr, [42, 0])


@pytest.mark.parametrize("trial", range(300))
def test_uniform_below_is_high_half_of_product(trial):
    rng = random.Random(trial)
    w = rng.getrandbits(64)
    n = rng.choice([1, 2, 3, 10, 25, rng.getrandbits(31) + 1, rng.getrandbits(63) + 1, M64])
    r = oracle.uniform_below(w, n)
    assert r == (w * n) >> 64
    assert 0 <= r < n


def test_uniform_below_extremes():
    assert oracle.uniform_below(0, 17) == 0
    assert oracle.uniform_below(M64, 17) == 16
    assert oracle.uniform_below(1 << 63, 10) == 5
    assert oracle.uniform_below(M64, 1) == 0


@pytest.mark.parametrize("seed,v,m,l", [(0, 0, 0, 0), (0, 5, 3, 1), (7, 8388607, 255, 2),
                                        (123456789, 2**31 - 1, 10**12, 7)])
def test_draw_word_keying(seed, v, m, l):
    for i in range(13):
        block = numpy_philox([i >> 2, v, m, l], [seed, 0])
        assert oracle.draw_word(seed, v, m, l, i) == block[i & 3]

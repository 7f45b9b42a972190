"""Pins of the oracle's subset sampler.

Floyd's algorithm (Bentley and Floyd, CACM 1987) draws d_i uniformly in
[0, n-k+i] for i = 0..k-1.  Over all prod_i (n-k+i+1) = n!/(n-k)! equally likely
draw sequences, every k-subset of [0, n) must come out exactly k! times: the
sampler is exactly uniform without replacement.  This is checked exhaustively
for n <= 7, every k.  The full composition (Philox words -> multiply-shift ->
Floyd) is checked statistically with a chi-square test.
"""
import itertools
import math
from collections import Counter

import pytest
from scipy import stats

import oracle


@pytest.mark.parametrize("n", range(0, 8))
def test_floyd_exact_uniformity_exhaustive(n):
    for k in range(0, n + 1):
        ranges = [range(n - k + i + 1) for i in range(k)]
        counts = Counter()
        for draws in itertools.product(*ranges):
            s = oracle.floyd_from_draws(n, k, list(draws))
            assert s == sorted(s)
            assert len(set(s)) == k
            assert all(0 <= x < n for x in s)
            counts[tuple(s)] += 1
        assert len(counts) == math.comb(n, k)
        assert set(counts.values()) == {math.factorial(k)}


def test_floyd_rejects_out_of_range_draw():
    with pytest.raises(ValueError):
        oracle.floyd_from_draws(5, 2, [4, 0])      # first draw must be in [0, 3]


def test_take_all_when_degree_not_above_fanout():
    for deg in range(0, 12):
        for f in (deg, deg + 1, 50):
            assert oracle.sample_positions(deg, f, 0, 3, 1, 0) == list(range(deg))


def test_zero_fanout_is_empty():
    assert oracle.sample_positions(40, 0, 0, 3, 1, 0) == []


def test_sampler_chi_square_degree6_k3():
    # C(6,3) = 20 cells, 1e5 independent keys (distinct node ids)
    counts = Counter()
    trials = 100000
    for v in range(trials):
        counts[tuple(oracle.sample_positions(6, 3, 99, v, 0, 0))] += 1
    assert len(counts) == 20
    obs = [counts[c] for c in sorted(counts)]
    chi2, p = stats.chisquare(obs)
    assert p > 1e-4, (chi2, p)


def test_sampler_marginals_degree40_k10():
    # every position equally likely: expected count trials * k / n
    trials, n, k = 40000, 40, 10
    hits = [0] * n
    for m in range(trials):
        for p in oracle.sample_positions(n, k, 5, 17, m, 1):
            hits[p] += 1
    chi2, p = stats.chisquare(hits)
    assert p > 1e-4, (chi2, p)


def test_sampler_depends_on_every_key_field():
    base = oracle.sample_positions(1000, 10, 1, 2, 3, 0)
    assert oracle.sample_positions(1000, 10, 1, 2, 3, 0) == base
    assert oracle.sample_positions(1000, 10, 2, 2, 3, 0) != base      # seed
    assert oracle.sample_positions(1000, 10, 1, 5, 3, 0) != base      # node
    assert oracle.sample_positions(1000, 10, 1, 2, 4, 0) != base      # minibatch
    assert oracle.sample_positions(1000, 10, 1, 2, 3, 1) != base      # hop

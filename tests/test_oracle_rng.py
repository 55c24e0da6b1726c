"""Pins of the oracle's counter-based draw (the reading of RandomNode /
UniformChoice of Algorithm 1, Section 3.3): SplitMix64's published outputs
and uniformity of the index it yields."""
import numpy as np
import pytest
from scipy.stats import chisquare

import oracle
from conftest import read_golden

GAMMA = 0x9E3779B97F4A7C15


def test_splitmix64_published_vectors():
    rows = read_golden("splitmix64_vectors.txt")
    assert len(rows) >= 6
    for seed, k, want in rows:
        state = (int(seed) + int(k) * GAMMA) % 2**64
        assert oracle.splitmix64(state) == int(want)


def test_pick_in_range_and_covers_all_values():
    key = oracle.rng_key(7, 3)
    for cnt in range(1, 34):
        ks = {oracle.pick(key, p, s, cnt) for p in range(40 * cnt) for s in (0, 1)}
        assert ks == set(range(cnt))


@pytest.mark.parametrize("cnt", [2, 3, 5, 7, 8, 16, 31, 32])
@pytest.mark.parametrize("stream", [0, 1])
def test_pick_uniform_chi2(cnt, stream):
    """10^5 draws for each candidate count, chi-square at the 1e-4 level."""
    key = oracle.rng_key(12345, 9)
    n = 100000
    ks = np.array([oracle.pick(key, p, stream, cnt) for p in range(n)])
    _, pval = chisquare(np.bincount(ks, minlength=cnt))
    assert pval > 1e-4


def test_streams_seeds_steps_decorrelated():
    """Node and rank draws of one pair, and draws of different steps or
    seeds, must not coincide systematically."""
    n, cnt = 100000, 8
    k1 = oracle.rng_key(1, 0)
    a = np.array([oracle.pick(k1, p, 0, cnt) for p in range(n)])
    b = np.array([oracle.pick(k1, p, 1, cnt) for p in range(n)])
    c = np.array([oracle.pick(oracle.rng_key(1, 1), p, 0, cnt) for p in range(n)])
    d = np.array([oracle.pick(oracle.rng_key(2, 0), p, 0, cnt) for p in range(n)])
    for other in (b, c, d):
        agree = np.mean(a == other)
        assert abs(agree - 1 / cnt) < 0.01
        # joint distribution of (a, other) is uniform over cnt*cnt cells
        _, pval = chisquare(np.bincount(a * cnt + other, minlength=cnt * cnt))
        assert pval > 1e-4

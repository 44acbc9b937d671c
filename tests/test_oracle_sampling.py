"""Pins of the oracle's neighbour sampling (CPU only).

Floyd's algorithm is pinned by brute force over every draw sequence; the
keyed sampler by chi-square uniformity over many keys and nodes.
"""
import itertools
import math

import numpy as np
import pytest
from scipy import stats


@pytest.mark.parametrize("d", range(1, 9))
def test_floyd_brute_force_exact_uniformity(orc, d):
    """Over all d!/(d-k)! draw sequences (t_i uniform in [0, d-k+i]) every
    k-subset of {0..d-1} comes out exactly k! times."""
    for k in range(0, d + 1):
        ranges = [range(d - k + i + 1) for i in range(k)]
        hist = {}
        total = 0
        for draws in itertools.product(*ranges):
            out = orc.floyd(d, k, list(draws))
            assert len(set(int(x) for x in out)) == k
            assert all(0 <= int(x) < d for x in out)
            key = tuple(sorted(int(x) for x in out))
            hist[key] = hist.get(key, 0) + 1
            total += 1
        assert total == math.perm(d, k)
        assert len(hist) == math.comb(d, k)
        assert set(hist.values()) == {math.factorial(k)}


def _subset_chi2(hist: np.ndarray, d: int, k: int):
    masks = [sum(1 << s for s in c) for c in itertools.combinations(range(d), k)]
    obs = hist[masks]
    assert obs.sum() == hist.sum(), "a sample outside the k-subsets of d"
    return stats.chisquare(obs).pvalue


@pytest.mark.parametrize("d,f,n", [(5, 2, 100000), (8, 3, 200000), (12, 5, 300000),
                                   (16, 15, 100000)])
def test_keyed_subsets_uniform_over_keys(pins, d, f, n):
    hist = np.zeros(1 << d, dtype=np.uint64)
    assert pins.pin_subset_hist(d, f, 17, 2, 1000, n, hist.ctypes.data) == 0
    assert _subset_chi2(hist, d, f) > 1e-4


@pytest.mark.parametrize("d,f,n", [(6, 3, 100000), (10, 4, 200000)])
def test_keyed_subsets_uniform_over_nodes(pins, d, f, n):
    hist = np.zeros(1 << d, dtype=np.uint64)
    assert pins.pin_subset_hist_nodes(d, f, 0, 1, 99, n, hist.ctypes.data) == 0
    assert _subset_chi2(hist, d, f) > 1e-4


def test_hub_marginals(pins):
    """A hub of in-degree 100,000 with fan-out 25: every slot is included
    with probability 25/100,000 (grouped into 100 bins of 1,000 slots)."""
    d, f, n = 100000, 25, 40000
    incl = np.zeros(d, dtype=np.uint64)
    assert pins.pin_marginals(d, f, 3, 0, 555, n, incl.ctypes.data) == 0
    assert incl.sum() == f * n
    bins = incl.reshape(100, 1000).sum(axis=1)
    assert stats.chisquare(bins).pvalue > 1e-4


def test_degree_at_most_fanout_takes_whole_row(orc):
    for d in range(0, 12):
        out = orc.sample_node(5, 9, 0, d, 11)
        assert list(out) == list(range(d))


def test_sample_node_invariants(orc):
    for seed in range(20):
        for d, f in [(20, 5), (100, 15), (16, 15), (1000, 25), (30, 29)]:
            s = orc.sample_node(seed, seed * 7 + 1, seed % 3, d, f)
            assert len(s) == min(d, f)
            assert np.all(np.diff(s.astype(np.int64)) > 0)
            assert s.max() < d


def test_different_layers_draw_independently(orc):
    a = [tuple(orc.sample_node(1, v, 0, 50, 5)) for v in range(200)]
    b = [tuple(orc.sample_node(1, v, 1, 50, 5)) for v in range(200)]
    assert sum(x == y for x, y in zip(a, b)) < 5

"""Seed batching (Section II-B: a mini-batch is a set of target vertices
drawn uniformly at random from the training set; Section III-E: each
trainer draws its batches from its own share of it).  The training set is a
seeded random subset of the vertices, each epoch shuffles it and cuts it
into consecutive batches of B, the last one partial and kept.  These tests
fix what that has to mean: a partition of the training set per epoch, the
batch sizes, determinism in the epoch seed, and uniformity of batch
membership (a fixed vertex lands in every batch index equally often, two
fixed vertices share a batch with probability (B-1)/(n-1), and every vertex
is equally likely to be in the training set)."""
import numpy as np
import pytest
from scipy import stats

import datagen
from datagen.configs import CONFIGS


@pytest.mark.parametrize("n, fraction, seed", [(1000, 0.08, 1), (2_449_029, 0.08, 304), (10, 0.5, 3), (7, 0.0, 2)])
def test_train_set_distinct_and_sized(n, fraction, seed):
    t = datagen.train_set(n, fraction, seed)
    assert t.dtype == np.int32
    assert len(t) == int(round(fraction * n))
    assert len(np.unique(t)) == len(t)
    assert t.size == 0 or (t.min() >= 0 and t.max() < n)


def test_workload_split_sizes():
    """The stated epoch shapes: 8% of 2,449,029 is 195,922 seeds, 196 batches
    of 1000 with a last one of 922; 1% of 111,059,956 is 1,110,600 seeds."""
    p = CONFIGS["products2m"]
    t = datagen.train_set(p.num_nodes, p.train_fraction, p.seeds[3])
    assert len(t) == 195_922
    b = datagen.epoch_batches(t, p.batch, p.seeds[3] + 1)
    assert len(b) == 196 and len(b[-1]) == 922
    big = CONFIGS["papers111m"]
    assert int(round(big.train_fraction * big.num_nodes)) == 1_110_600


@pytest.mark.parametrize("n_train, batch", [(100, 10), (1001, 64), (37, 37), (36, 40), (5, 1)])
def test_epoch_is_a_partition(n_train, batch):
    train = datagen.permutation(10 * n_train, 11)[:n_train]
    batches = datagen.epoch_batches(train, batch, 5)
    assert len(batches) == -(-n_train // batch)
    assert all(len(x) == batch for x in batches[:-1])
    assert len(batches[-1]) == n_train - batch * (len(batches) - 1) > 0
    joined = np.concatenate(batches)
    assert np.array_equal(np.sort(joined), np.sort(train))


def test_epoch_seed_determinism():
    train = datagen.train_set(5000, 0.2, 9)
    a = datagen.epoch_batches(train, 100, 17)
    b = datagen.epoch_batches(train, 100, 17)
    c = datagen.epoch_batches(train, 100, 18)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    assert not all(np.array_equal(x, y) for x, y in zip(a, c))
    assert datagen.batch_seed(0x1234, 5) == 0x1231


def test_batch_index_of_a_vertex_is_uniform():
    """Over many epoch seeds, a fixed vertex falls into each of the 5 batch
    indices equally often (chi-square, 4 degrees of freedom), and so does its
    position within the epoch (50 positions)."""
    train = np.arange(50, dtype=np.int32)
    epochs = 5000
    idx = np.zeros((3, 5), np.int64)
    pos = np.zeros(50, np.int64)
    for e in range(epochs):
        order = np.concatenate(datagen.epoch_batches(train, 10, 1000 + e))
        where = np.empty(50, np.int64)
        where[order] = np.arange(50)
        for k, v in enumerate((0, 17, 49)):
            idx[k, where[v] // 10] += 1
        pos[where[0]] += 1
    for k in range(3):
        assert stats.chisquare(idx[k]).pvalue > 1e-4, idx[k]
    assert stats.chisquare(pos).pvalue > 1e-4


def test_pair_shares_a_batch_with_the_right_probability():
    """Two fixed vertices are in the same batch with probability
    (B - 1) / (n - 1) when batches are uniform random subsets."""
    n, B, epochs = 40, 8, 6000
    train = np.arange(n, dtype=np.int32)
    hits = 0
    for e in range(epochs):
        for b in datagen.epoch_batches(train, B, 7 + e):
            if 3 in b and 21 in b:
                hits += 1
    p = (B - 1) / (n - 1)
    sd = np.sqrt(epochs * p * (1 - p))
    assert abs(hits - epochs * p) < 5 * sd, (hits, epochs * p)


def test_training_set_membership_is_uniform():
    """Every vertex is equally likely to be drawn into the training set."""
    n, k, trials = 20, 5, 4000
    count = np.zeros(n, np.int64)
    for s in range(trials):
        count[datagen.train_set(n, k / n, 50 + s)] += 1
    assert count.sum() == k * trials
    assert stats.chisquare(count).pvalue > 1e-4, count

"""Pins of the oracle's random-number layer (CPU only).

Philox4x32-10 is pinned to the published known-answer vectors; the bounded
draw is pinned by enumerating every 32-bit word.
"""
import ctypes
import os

import numpy as np
import pytest
from scipy import stats

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat_rows():
    rows = []
    with open(GOLDEN) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            w = [int(x, 16) for x in line.split()]
            rows.append((w[0:4], w[4:6], w[6:10]))
    return rows


def test_philox_known_answers(orc):
    rows = _kat_rows()
    assert len(rows) == 3
    for ctr, key, want in rows:
        got = orc.philox4x32_10(ctr, key)
        assert [int(x) for x in got] == want, (ctr, key)


def test_philox_counter_and_key_sensitivity(orc):
    base = orc.philox4x32_10([1, 2, 3, 4], [5, 6])
    for i in range(4):
        c = [1, 2, 3, 4]
        c[i] ^= 1
        assert not np.array_equal(orc.philox4x32_10(c, [5, 6]), base)
    for i in range(2):
        k = [5, 6]
        k[i] ^= 1
        assert not np.array_equal(orc.philox4x32_10([1, 2, 3, 4], k), base)


@pytest.mark.parametrize("m", [1, 2, 3, 7, 10, 1000, 100003])
def test_bounded_draw_exhaustive(pins, m):
    """Every value in [0, m) is produced by exactly floor(2^32/m) words and
    exactly (2^32 mod m) words are rejected: the draw is exactly uniform."""
    counts = np.zeros(m, dtype=np.uint64)
    rejects = ctypes.c_uint64(0)
    bad = pins.pin_bounded_exhaustive(m, counts.ctypes.data, ctypes.byref(rejects), 8)
    assert bad == 0
    assert rejects.value == (1 << 32) % m
    assert np.all(counts == (1 << 32) // m)


def test_bounded_draw_small_cases(orc):
    # m = 1 always accepts 0; a power of two never rejects.
    for x in (0, 1, 0xFFFFFFFF, 0x80000000):
        assert orc.bounded_from_word(x, 1) == 0
        assert orc.bounded_from_word(x, 1 << 20) == x >> 12
    # m = 3: threshold (2^32 - 3) mod 3 = 1, so only x with lo32(3x) == 0, i.e. x = 0, is rejected.
    assert orc.bounded_from_word(0, 3) is None
    assert orc.bounded_from_word(1, 3) == 0
    assert orc.bounded_from_word(0xFFFFFFFF, 3) == 2


def test_uniform_below_retry_path_is_uniform(orc):
    """m = 2^31 + 1 rejects about half of all words, so all four words of a
    Philox block are rejected in ~1/16 of draws and the retry counter is
    exercised; the result must stay uniform."""
    m = (1 << 31) + 1
    n = 40000
    vals = np.array([orc.uniform_below(7, v, 3, 1, m) for v in range(n)], dtype=np.uint64)
    assert vals.max() < m
    bins = np.bincount((vals * 16 // m).astype(np.int64), minlength=16)
    p = stats.chisquare(bins).pvalue
    assert p > 1e-4, (bins, p)


def test_uniform_below_is_a_pure_function(orc):
    a = [orc.uniform_below(123, 5, 1, i, 1000) for i in range(50)]
    b = [orc.uniform_below(123, 5, 1, i, 1000) for i in range(50)]
    assert a == b
    c = [orc.uniform_below(124, 5, 1, i, 1000) for i in range(50)]
    assert a != c

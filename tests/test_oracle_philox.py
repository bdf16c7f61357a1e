"""Pins for the oracle's Philox4x32-10 (published known-answer vectors) and
the u = ((w >> 8) | 1) * 2^-24 map."""
import os

import numpy as np

from oracle.philox import philox4x32_10, philox_words, u24_odd

GOLD = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat():
    rows = []
    for line in open(GOLD):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        v = [int(x, 16) for x in line.split()]
        rows.append((v[0:4], v[4:6], v[6:10]))
    return rows


def test_known_answer_vectors():
    rows = _kat()
    assert len(rows) == 3
    for ctr, key, out in rows:
        got = [int(x) for x in philox4x32_10(*ctr, *key)]
        assert got == out


def test_vectorised_matches_scalar():
    ctr = np.arange(1000, dtype=np.uint64) * 2654435761 % (1 << 32)
    a = philox4x32_10(ctr, 7, 9, 11, 123, 456)
    for i in (0, 17, 999):
        b = philox4x32_10(int(ctr[i]), 7, 9, 11, 123, 456)
        assert [int(x[i]) for x in a] == [int(x) for x in b]


def test_word_selection_and_seed_split():
    idx = np.arange(8, dtype=np.uint64)
    w = philox_words(idx, 5, 6, 7, (3 << 32) | 9)
    b0 = philox4x32_10(0, 5, 6, 7, 9, 3)
    b1 = philox4x32_10(1, 5, 6, 7, 9, 3)
    assert [int(x) for x in w] == [int(x) for x in b0] + [int(x) for x in b1]


def test_u24_odd_exact_and_open_interval():
    w = np.array([0, 0xFF, 0x100, 0xFFFFFFFF, 0x80000000], dtype=np.uint32)
    u = u24_odd(w)
    assert u.dtype == np.float32
    exp = np.array([1, 1, 1, (1 << 24) - 1, (1 << 23) | 1], dtype=np.float64) / (1 << 24)
    assert np.array_equal(u.astype(np.float64), exp)
    assert (u > 0).all() and (u < 1).all()


def test_uniformity_chi_square():
    idx = np.arange(1 << 20, dtype=np.uint64)
    u = u24_odd(philox_words(idx, 1, 2, 3, 42)).astype(np.float64)
    counts, _ = np.histogram(u, bins=64, range=(0, 1))
    expct = len(u) / 64
    chi2 = ((counts - expct) ** 2 / expct).sum()
    # 63 dof: the 99.99% quantile is about 117
    assert chi2 < 117
    assert abs(u.mean() - 0.5) < 2e-3


def test_range_equals_per_word_evaluation():
    """philox_range evaluates each counter block once; it must give exactly
    the words philox_words gives element by element."""
    import numpy as np
    from oracle.philox import philox_range, philox_words
    for start, n, seed in ((0, 1, 5), (0, 13, 7), (4096, 1000, 3), (1 << 24, 4097, 1 << 40)):
        a = philox_range(start, n, 9, 2, 1, seed)
        b = philox_words(np.arange(start, start + n, dtype=np.uint64), 9, 2, 1, seed)
        assert np.array_equal(a, b)

"""Pins for the oracle's group advantages (Eq. 2) and the dual-end group mean (Eq. 3)."""
import numpy as np
import pytest

from oracle.advantage import group_advantages, kept_advantages, dual_group_mean


def test_matches_numpy_mean_and_std():
    rng = np.random.default_rng(0)
    for _ in range(200):
        k = int(rng.integers(1, 33))
        r = rng.normal(0, 2, k)
        a = group_advantages(list(r), eps=0.0 if r.std() > 0 else 1e-6)
        exp = (r - r.mean()) / (r.std() if r.std() > 0 else 1e-6)
        assert np.allclose(a, exp, rtol=1e-12, atol=1e-12)


def test_closed_forms():
    rng = np.random.default_rng(1)
    for _ in range(100):
        k = int(rng.integers(2, 17))
        r = rng.integers(0, 2, k).astype(float)
        if r.min() == r.max():
            assert group_advantages(list(r)) == [0.0] * k
            continue
        a = np.array(group_advantages(list(r), eps=0.0))
        assert abs(a.sum()) < 1e-12
        assert (a ** 2).sum() == pytest.approx(k, rel=1e-12)
        # binary rewards: correct ones share one positive advantage sqrt((1-p)/p)
        p = r.mean()
        assert np.allclose(a[r == 1], np.sqrt((1 - p) / p), rtol=1e-12)
        assert np.allclose(a[r == 0], -np.sqrt(p / (1 - p)), rtol=1e-12)
    assert group_advantages([0.5]) == [0.0]


def test_affine_invariance():
    rng = np.random.default_rng(2)
    r = list(rng.normal(0, 1, 8))
    a = group_advantages(r, eps=0.0)
    b = group_advantages([3.5 * x - 7.0 for x in r], eps=0.0)
    assert np.allclose(a, b, rtol=1e-12, atol=1e-12)


def test_eq3_dual_group_mean():
    rng = np.random.default_rng(3)
    for _ in range(100):
        K, L = int(rng.integers(1, 15)), int(rng.integers(1, 4))
        rs, rl = list(rng.integers(0, 2, K).astype(float)), list(rng.integers(0, 2, L).astype(float))
        assert dual_group_mean(rs, rl) == pytest.approx(np.mean(rs + rl), rel=1e-12, abs=1e-15)
    # with K >> L the group mean is anchored at the short side's mean (the paper's approximation)
    assert abs(dual_group_mean([1.0] * 31, [0.0]) - 1.0) <= 1 / 32


def test_kept_advantages_maps_groups():
    kept = {0: [3, 1], 1: [4, 6]}
    rew = {1: 1.0, 3: 0.0, 4: 2.0, 6: 2.0}
    a = kept_advantages(kept, rew)
    assert a[0] == pytest.approx([-1.0, 1.0], abs=1e-5) and a[1] == [0.0, 0.0]

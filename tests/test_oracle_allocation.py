"""Pins for the oracle's adaptive redundancy allocation (Alg. 1, App. B):
the hand-worked examples, brute-force minimisation of the objective, the
closed-form budget against a direct search of the utility, and invariants."""
import itertools
import json
import math
import os
import random

import numpy as np
import pytest

from oracle.allocation import (allocate, objective, redundancy_budget, minmax_norm, length_std,
                               ema_update, fill_unseen, dataset_rho, marginal_gain)

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "allocation_example.json")))


@pytest.mark.parametrize("case", GOLD["budget"]["cases"])
def test_budget_worked_example(case):
    b = GOLD["budget"]
    assert redundancy_budget(case["rho"], case["lambda"], case["k_cost"], b["n_prompts"], b["M"]) \
        == case["m_total"]


@pytest.mark.parametrize("ex", GOLD["allocation"])
def test_allocation_worked_example(ex):
    assert minmax_norm(ex["sigma"]) == pytest.approx(ex["weights"], abs=0)
    got = allocate(ex["sigma"], ex["m_total"], ex["m_low"], ex["m_up"])
    assert got == ex["alloc"]
    assert objective(ex["sigma"], got) == pytest.approx(ex["objective"], rel=1e-15)
    modes = ["short" if a >= ex["m_up"] else "dual" for a in got]
    assert modes == ex["modes"]


def _brute(sigma, total, lo, hi):
    best = math.inf
    for alloc in itertools.product(range(lo, hi + 1), repeat=len(sigma)):
        if sum(alloc) == total:
            best = min(best, objective(sigma, alloc))
    return best


def test_greedy_reaches_brute_force_optimum():
    """The objective is separable and convex in each M'_i, so the greedy
    must attain the minimum found by enumerating every feasible allocation."""
    rng = random.Random(7)
    for _ in range(300):
        n = rng.randint(1, 5)
        lo = rng.randint(1, 4)
        hi = lo + rng.randint(0, 4)
        sigma = [rng.choice([0.0, 1.0, 2.5, 3.0, rng.random() * 100]) for _ in range(n)]
        total = rng.randint(n * lo, n * hi)
        got = allocate(sigma, total, lo, hi)
        assert sum(got) == total and all(lo <= a <= hi for a in got)
        assert objective(sigma, got) == pytest.approx(_brute(sigma, total, lo, hi), rel=1e-12, abs=1e-15)


def test_invariants_and_monotonicity():
    rng = np.random.default_rng(3)
    for _ in range(50):
        n = int(rng.integers(2, 40))
        sigma = list(rng.lognormal(5, 1, n))
        M = int(rng.integers(2, 9))
        total = int(rng.integers(n * M, 2 * n * M + 1))
        got = allocate(sigma, total, M, 2 * M)
        assert sum(got) == total
        assert all(M <= a <= 2 * M for a in got)
        # a prompt with a larger spread never gets fewer candidates
        for i in range(n):
            for j in range(n):
                if sigma[i] > sigma[j]:
                    assert got[i] >= got[j]


def test_budget_above_capacity_and_degenerate_batches():
    assert allocate([1.0, 2.0], 100, 2, 4) == [4, 4]      # surplus stays unallocated
    assert allocate([], 10, 2, 4) == []
    assert allocate([5.0], 3, 2, 4) == [3]
    assert allocate([1.0, 2.0], 4, 2, 4) == [2, 2]        # nothing to hand out


def test_budget_maximises_the_utility():
    """App. B: the integer maximiser of U(M) = rho ln M - lambda (k M + c) on
    [M N, 2 M N] is floor(M*) or floor(M*)+1 (U is concave); the closed form
    takes floor(M*) and clips."""
    rng = np.random.default_rng(11)
    for _ in range(200):
        rho, lam, kc = rng.uniform(0.1, 3), rng.uniform(1e-3, 0.1), rng.uniform(0.1, 20)
        N, M = int(rng.integers(1, 64)), int(rng.integers(1, 16))
        lo, hi = M * N, 2 * M * N
        grid = np.arange(lo, hi + 1)
        U = rho * np.log(grid) - lam * kc * grid
        best = int(grid[int(np.argmax(U))])
        got = redundancy_budget(rho, lam, kc, N, M)
        assert lo <= got <= hi
        assert abs(got - best) <= 1
        star = rho / (lam * kc)
        if star <= lo:
            assert got == lo and best == lo
        if star >= hi + 1:
            assert got == hi and best == hi


def test_length_statistics():
    rng = np.random.default_rng(5)
    for _ in range(20):
        x = rng.integers(1, 5000, int(rng.integers(1, 40)))
        assert length_std(list(x)) == pytest.approx(float(np.std(x)), rel=1e-12, abs=1e-12)
        assert dataset_rho(list(x)) == pytest.approx(float(np.std(x) / np.mean(x)), rel=1e-12)
    assert length_std([3, 3, 3]) == 0.0


def test_ema_and_unseen_prompts():
    v, s = [0.0, 0.0, 0.0], [False, False, False]
    v, s = ema_update(v, s, [4.0, None, 2.0])
    assert v == [4.0, 0.0, 2.0] and s == [True, False, True]
    v, s = ema_update(v, s, [8.0, 6.0, None])
    assert v == [6.0, 6.0, 2.0]
    # constant observations are a fixed point; alpha = 1 keeps the last value
    w, t = ema_update([3.0], [True], [3.0])
    assert w == [3.0]
    w, t = ema_update([3.0], [True], [9.0], alpha=1.0)
    assert w == [9.0]
    assert fill_unseen([1.0, 0.0, 3.0], [True, False, True]) == [1.0, 2.0, 3.0]
    assert fill_unseen([0.0], [False]) == [0.0]


def test_marginal_gain_is_the_objective_decrease():
    for w in (0.0, 0.3, 1.0):
        for m in range(1, 20):
            assert marginal_gain(w, m) == pytest.approx(w / m - w / (m + 1), rel=1e-14, abs=1e-300)

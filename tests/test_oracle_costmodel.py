"""Pins for the oracle's rollout cost model (Eq. 4) and PTL fit (App. A):
a step-by-step simulation of the decode loop, closed forms, and exact
recovery of a known three-stage curve."""
import numpy as np
import pytest

from oracle.costmodel import ptl_eval, rollout_cost, rollout_cost_dp, fit_ptl


def _simulate(lengths, ptl):
    """The decode loop itself: at step t every response with length >= t runs."""
    T = 0.0
    for t in range(1, max(lengths) + 1):
        b = sum(1 for l in lengths if l >= t)
        T += ptl(b)
    return T


def test_eq4_equals_step_simulation():
    rng = np.random.default_rng(1)
    ptl = lambda b: 3.0 + 0.25 * b + 0.01 * max(0, b - 5) ** 1.5
    for _ in range(200):
        n = int(rng.integers(1, 30))
        lengths = list(rng.integers(0, 60, n))
        assert rollout_cost(lengths, ptl) == pytest.approx(_simulate(lengths, ptl) if max(lengths) else 0.0,
                                                           rel=1e-12, abs=1e-12)


def test_eq4_closed_forms():
    lengths = [5, 9, 2, 14, 14, 7]
    assert rollout_cost([8] * 6, lambda b: 2.0 + b) == 8 * (2.0 + 6)          # equal lengths
    assert rollout_cost(lengths, lambda b: 4.0) == 4.0 * max(lengths)            # constant PTL
    assert rollout_cost(lengths, lambda b: 0.5 * b) == pytest.approx(0.5 * sum(lengths))  # linear PTL
    assert rollout_cost([], lambda b: 1.0) == 0.0
    assert rollout_cost_dp([[3, 4], [10], []], lambda b: 1.0) == 10.0


def test_fit_recovers_a_three_stage_curve():
    true = (64.0, 256.0, 2.0, 0.004, 0.010, 0.020)
    b = np.array([1, 2, 4, 8, 16, 32, 48, 64, 96, 128, 160, 200, 256, 300, 384, 448, 512] * 2, float)
    y = np.array([ptl_eval(true, x) for x in b])
    p = fit_ptl(b, y)
    assert p[0] == 64.0 and p[1] == 256.0
    assert np.allclose(p[2:], true[2:], rtol=1e-9, atol=1e-12)
    # noisy samples: the fit's residual is no larger than the true curve's
    rng = np.random.default_rng(3)
    yn = y + rng.normal(0, 0.05, len(y))
    q = fit_ptl(b, yn)
    sse = lambda prm: float(sum((yn[i] - ptl_eval(prm, b[i])) ** 2 for i in range(len(b))))
    assert sse(q) <= sse(true) + 1e-12
    # continuity: the three pieces meet at the breakpoints
    for bp in q[:2]:
        assert ptl_eval(q, bp - 1e-9) == pytest.approx(ptl_eval(q, bp + 1e-9), abs=1e-6)


def test_fit_degenerate_inputs():
    p = fit_ptl([8, 8, 8], [1.0, 2.0, 3.0])
    assert ptl_eval(p, 8) == pytest.approx(2.0)
    p = fit_ptl([4, 8], [1.0, 2.0])
    assert ptl_eval(p, 4) == pytest.approx(1.0) and ptl_eval(p, 8) == pytest.approx(2.0)


def test_fit_with_intercept_preserves_the_total():
    """Least squares with an intercept leaves residuals summing to zero, so
    Eq. 4 with the fitted curve reproduces the measured total of the very
    steps it was fitted on (the identity the engine's step accounting is
    checked with)."""
    rng = np.random.default_rng(5)
    lengths = list(rng.integers(1, 400, 64))
    steps = [(t, sum(1 for l in lengths if l >= t)) for t in range(1, max(lengths) + 1)]
    lat = [1.0 + 0.01 * b + rng.normal(0, 0.1) for _, b in steps]
    p = fit_ptl([b for _, b in steps], lat)
    assert rollout_cost(lengths, lambda b: ptl_eval(p, b)) == pytest.approx(sum(lat), rel=1e-9)

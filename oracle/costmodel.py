"""Rollout cost model (paper Sec. 4.2.1, Eq. 4) and the per-token latency
curve it uses (App. A).  TEST INFRASTRUCTURE: the plain statement of what the
library's cost-model entry points compute.

* Eq. 4: for responses with sorted lengths l_[1] <= ... <= l_[n] (l_[0] = 0)
  decoded together, T = sum_m (l_[m] - l_[m-1]) * PTL(n - m + 1): between two
  consecutive completions every still-running response costs one step whose
  latency depends on how many are running.
* Data parallel: the batch cost is the maximum over groups.
* PTL: a continuous three-stage piecewise-linear function of the batch size,
  PTL(b) = c0 + c1 b + c2 max(0, b - b1) + c3 max(0, b - b2), b1 < b2, fitted
  by least squares to measured (batch size, step latency) pairs.

Readings (listed in the design notes): with xs the D distinct measured batch
sizes in increasing order, the breakpoints range over b1 = xs[i], b2 = xs[j],
1 <= i < j <= D-2, the pairs for which every piece is determined by the data
(two sizes at or below b1, one in (b1, b2], one above b2); least squares on
the coefficients for each pair, the smallest residual wins, ties to the first
pair in (i, j) lexicographic order.  With fewer than four distinct sizes the
curve is one least-squares line (b1 = b2 = the largest size, c2 = c3 = 0;
a single size gives the mean latency).  On one GPU the "batch" of Eq. 4 is
all trajectories decoded together; their lengths are the numbers of decode
steps each took part in.

Pins (tests/test_oracle_costmodel.py): a direct step-by-step simulation of the
decode loop, closed forms (equal lengths, constant and linear PTL), exact
recovery of a known curve from noiseless samples.
"""
import numpy as np


def ptl_eval(params, b):
    """params = (b1, b2, c0, c1, c2, c3)."""
    b1, b2, c0, c1, c2, c3 = params
    b = float(b)
    return c0 + c1 * b + c2 * max(0.0, b - b1) + c3 * max(0.0, b - b2)


def rollout_cost(lengths, ptl):
    """Eq. 4 over one batch; ptl is a callable of the batch size."""
    ls = sorted(int(x) for x in lengths)
    n = len(ls)
    T, prev = 0.0, 0
    for m in range(1, n + 1):
        T += (ls[m - 1] - prev) * ptl(n - m + 1)
        prev = ls[m - 1]
    return T


def rollout_cost_dp(groups, ptl):
    """Data parallel: the slowest group sets the batch cost."""
    return max((rollout_cost(g, ptl) for g in groups), default=0.0)


def _design(b, b1, b2):
    b = np.asarray(b, dtype=np.float64)
    return np.stack([np.ones_like(b), b, np.maximum(0.0, b - b1), np.maximum(0.0, b - b2)], axis=1)


def fit_ptl(bsz, lat):
    """Least-squares three-stage fit; returns (b1, b2, c0, c1, c2, c3)."""
    bsz = np.asarray(bsz, dtype=np.float64)
    lat = np.asarray(lat, dtype=np.float64)
    xs = np.unique(bsz)
    D = len(xs)
    if D == 0:
        return (0.0, 0.0, 0.0, 0.0, 0.0, 0.0)
    if D == 1:
        return (float(xs[0]), float(xs[0]), float(np.mean(lat)), 0.0, 0.0, 0.0)
    if D < 4:
        X = np.stack([np.ones_like(bsz), bsz], axis=1)
        coef, *_ = np.linalg.lstsq(X, lat, rcond=None)
        return (float(xs[-1]), float(xs[-1]), float(coef[0]), float(coef[1]), 0.0, 0.0)
    best, best_p = None, None
    for i in range(1, D - 2):
        for j in range(i + 1, D - 1):
            b1, b2 = xs[i], xs[j]
            X = _design(bsz, b1, b2)
            coef, *_ = np.linalg.lstsq(X, lat, rcond=None)
            r = lat - X @ coef
            sse = float(r @ r)
            if best is None or sse < best:
                best, best_p = sse, (float(b1), float(b2), *[float(c) for c in coef])
    return best_p

"""Adaptive redundancy allocation (paper Sec. 4.2.2, App. B, App. C / Alg. 1).
TEST INFRASTRUCTURE: the plain statement of what the library's allocation
entry points compute.

* Per-prompt long-tail signal: the standard deviation of the response lengths
  of the prompt's candidates, smoothed over rollouts by an exponential moving
  average (Sec. 4.2.2 "smoothed historical variance", App. C "EMA").
* Alg. 1: weights w_i = Norm(sigma_i) (min-max over the batch), every prompt
  starts at M_low, and the remaining budget is handed out one unit at a time
  to the prompt with the largest marginal gain
  w_i * (1/M'_i - 1/(M'_i + 1)) among those still below M_up.
* App. B: the total budget maximises rho * ln(M) - lambda * (k * M + c), so
  M* = rho / (lambda * k), floored and clipped to [M*N, 2*M*N].

Readings where the paper is silent (listed in the design notes):
* Norm of a batch whose values are all equal gives every weight 1.
* argmax ties go to the lowest prompt index; gains are compared as float64
  values computed exactly as written above.
* The EMA rate is alpha = 0.5; a prompt seen for the first time takes its
  observed value; a prompt never observed takes the mean over observed ones.
* The observed length spread of a prompt is the population standard
  deviation of the lengths its candidates reached in the rollout (aborted
  candidates at the length they had when aborted).
* If the budget exceeds N * M_up the surplus stays unallocated.

Pins (tests/test_oracle_allocation.py): brute-force minimisation of the
objective over every feasible allocation for small batches (the objective is
separable and convex, so the greedy must reach the optimum), the closed form
and its clip, a hand-worked example (tests/golden/allocation_example.json),
and invariants (sum, bounds, monotone in the weight).
"""
import math


def minmax_norm(values):
    """Min-max normalisation over the batch (Sec. 4.2.2); all equal -> 1."""
    lo, hi = min(values), max(values)
    if hi == lo:
        return [1.0 for _ in values]
    return [(float(v) - lo) / (hi - lo) for v in values]


def marginal_gain(w, m):
    """Objective decrease w/m - w/(m+1) of one more candidate (Alg. 1)."""
    return w * (1.0 / m - 1.0 / (m + 1))


def allocate(sigma, m_total, m_low, m_up):
    """Alg. 1: greedy allocation of m_total candidates over the prompts."""
    n = len(sigma)
    if n == 0:
        return []
    w = minmax_norm(sigma)
    alloc = [m_low] * n
    remain = m_total - n * m_low
    while remain > 0:
        best, best_i = None, -1
        for i in range(n):
            if alloc[i] >= m_up:
                continue
            d = marginal_gain(w[i], alloc[i])
            if best is None or d > best:
                best, best_i = d, i
        if best_i < 0:
            break
        alloc[best_i] += 1
        remain -= 1
    return alloc


def objective(sigma, alloc):
    """sum_i Norm(sigma_i) / M'_i (the quantity Alg. 1 minimises)."""
    return sum(w / m for w, m in zip(minmax_norm(sigma), alloc))


def redundancy_budget(rho, lam, k_cost, n_prompts, M):
    """App. B: U(M) = rho ln M - lambda (k M + c) is maximal at M* = rho/(lambda k);
    M_total = clip(floor(M*), M N, 2 M N)."""
    lo, hi = M * n_prompts, 2 * M * n_prompts
    if not (lam > 0 and k_cost > 0):
        return hi
    star = rho / (lam * k_cost)
    if not math.isfinite(star):
        return hi if star > 0 else lo
    return int(min(max(math.floor(star), lo), hi))


def length_std(lengths):
    """Population standard deviation of one prompt's candidate lengths."""
    n = len(lengths)
    if n == 0:
        return 0.0
    mu = sum(float(x) for x in lengths) / n
    return math.sqrt(sum((float(x) - mu) ** 2 for x in lengths) / n)


def ema_update(prev, seen, observed, alpha=0.5):
    """Smoothed per-prompt statistic.  prev/seen: current estimates and flags
    (None entries of `observed` mean "not rolled out this time")."""
    out, out_seen = list(prev), list(seen)
    for i, o in enumerate(observed):
        if o is None:
            continue
        out[i] = float(o) if not seen[i] else alpha * float(o) + (1.0 - alpha) * prev[i]
        out_seen[i] = True
    return out, out_seen


def fill_unseen(values, seen):
    """Prompts never observed take the mean of the observed ones (0 if none)."""
    obs = [v for v, s in zip(values, seen) if s]
    mean = sum(obs) / len(obs) if obs else 0.0
    return [v if s else mean for v, s in zip(values, seen)]


def dataset_rho(lengths):
    """rho = sigma_L / mean_L over all response lengths (App. B)."""
    n = len(lengths)
    mu = sum(float(x) for x in lengths) / n
    return length_std(lengths) / mu if mu > 0 else 0.0

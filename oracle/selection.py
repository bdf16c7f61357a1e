"""Distribution-aware trajectory selection (paper Sec. 4.1.2, Sec. 4.3.1, Alg. 2).

Per prompt q_i with candidate pool T_i of M'_i = m trajectories, target group
size M = k, dual-end short size K = k - L (L = 1 as in the paper's main runs):

* Dual-end length sampling (Alg. 2, M'_i < M_up): once every candidate is
  finished, Y_i = Y_short (top-K shortest) U Y_long (top-L longest), where the
  longest side excludes trajectories that hit the system length limit.
* Tail pruning with proactive early stopping (Alg. 2, M'_i >= M_up): keep the
  top-M shortest; generation stops as soon as M valid complete responses exist,
  and the remaining M'_i - M candidates are pruned (aborted).

Readings where the paper is silent (each listed in the design notes):
* valid = ended by end-of-sequence at length <= cap; truncated = reached cap.
* Order "shortest first" (<_short): key (truncated, length, -mean_logprob, id)
  ascending; mean log-prob descending ("certain" first) breaks length ties,
  then the trajectory id.  NaN mean log-prob sorts as -inf; -0 equals +0.
* Order "longest first" (<_long, valid members only): key (-length,
  -mean_logprob, id) ascending.
* Fewer than M valid members: fill with the remaining members in <_short order
  (so exactly M are always kept).
* Dual-end: short side first, long side from the remaining valid members,
  any deficit filled from the remaining members in <_short order.

Pins: brute-force enumeration of all k-subsets on small groups, the hand-worked
two-prompt example (tests/golden/appendix_example.json), and invariants
(exactly k kept, kept within the group, early-stop kept set equal to the
offline kept set, independence of processing order).
"""
import math

LIVE, EOS, TRUNC, ABORTED = 0, 1, 2, 3


def nk(x: float) -> float:
    """-x with NaN mapped to +inf and -0 to +0."""
    if x != x:
        return math.inf
    y = -float(x)
    return 0.0 if y == 0.0 else y


def key_short(t):
    """t: dict with g, length, trunc (bool), mean_lp."""
    return (1 if t["trunc"] else 0, t["length"], nk(t["mean_lp"]), t["g"])


def key_long(t):
    return (-t["length"], nk(t["mean_lp"]), t["g"])


def select_short(members, k):
    """Top-k under <_short (valid first, then truncated fill)."""
    return [t["g"] for t in sorted(members, key=key_short)[:k]]


def select_dual(members, k, L):
    K = k - L
    ordered = sorted(members, key=key_short)
    y_short = ordered[:K]
    taken = {t["g"] for t in y_short}
    rest_valid = [t for t in members if (t["g"] not in taken) and not t["trunc"]]
    y_long = sorted(rest_valid, key=key_long)[:L]
    taken |= {t["g"] for t in y_long}
    fill = [t for t in ordered if t["g"] not in taken][:k - len(y_short) - len(y_long)]
    return [t["g"] for t in y_short] + [t["g"] for t in y_long] + [t["g"] for t in fill]


def group_decision(members, k, L, m_up, early_stop=True):
    """Decide whether a group completes now.

    members: list of dicts with g, status (LIVE/EOS/TRUNC), length, trunc, mean_lp.
    Returns (complete: bool, kept: list[int], abort: list[int]).
    """
    m = len(members)
    live = [t for t in members if t["status"] == LIVE]
    done = [t for t in members if t["status"] != LIVE]
    if m >= m_up:
        valid = [t for t in done if t["status"] == EOS]
        if early_stop and len(valid) >= k:
            return True, select_short(valid, k), [t["g"] for t in live]
        if not live:
            return True, select_short(done, k), []
        return False, [], []
    if live:
        return False, [], []
    return True, select_dual(done, k, L), []


def reclaimed_pages(page_lists, completed, m):
    """KV page ids a selection frees: for every group that completed (ascending
    group index), the page lists of its members j = 0 .. m-1 in member order
    (at completion every member is done: finished, or aborted by the early
    stop, and all their pages return to the pool; Alg. 2's abort, Sec. 4.3.1).
    page_lists[g]: the pages trajectory g = i*m + j holds."""
    out = []
    for i in sorted(completed):
        for j in range(m):
            out.extend(int(p) for p in page_lists[i * m + j])
    return out

"""Pins for the oracle's selection (Alg. 2): the hand-worked example,
brute-force enumeration of k-subsets, and invariants."""
import itertools
import json
import os
import random

import numpy as np
import pytest

from oracle.selection import (LIVE, EOS, TRUNC, ABORTED, group_decision, select_short,
                              select_dual, key_short, nk)
from oracle.rollout import schedule_only

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "appendix_example.json")))
_ST = {"eos": EOS, "trunc": TRUNC, "aborted": ABORTED}


def _run(ex, m_up, early_stop=True, draws=None, mlp=None, m=None, k=None, cap=None):
    draws = ex["draws"] if draws is None else draws
    mlp = ex["mean_lp"] if mlp is None else mlp
    m = ex["m"] if m is None else m
    k = ex["k"] if k is None else k
    cap = ex["cap"] if cap is None else cap
    P = len(draws) // m
    return schedule_only(draws, P, m, k, cap, ex["prompt_len"], L=ex["L"], m_up=m_up,
                         page=ex["page_size"], early_stop=early_stop,
                         mean_lp=np.asarray(mlp, np.float32))


def test_appendix_short_mode():
    ex = GOLD
    r = _run(ex, ex["short"]["m_up"])
    exp = ex["short"]
    assert {str(i): v for i, v in r["kept"].items()} == exp["kept"]
    assert {str(i): v for i, v in r["done_step"].items()} == exp["done_step"]
    assert r["steps"] == exp["steps"]
    assert r["tokens_decoded"] == exp["tokens_decoded"]
    assert r["pages_hwm"] == exp["pages_hwm"]
    assert r["pages_end"] == exp["pages_end"]
    assert r["length"] == exp["lengths"]
    assert r["status"] == [_ST[s] for s in exp["status"]]


def test_appendix_no_abort_and_dual():
    ex = GOLD
    r = _run(ex, ex["no_abort"]["m_up"], early_stop=False)
    assert r["steps"] == ex["no_abort"]["steps"]
    assert r["tokens_decoded"] == ex["no_abort"]["tokens_decoded"]
    assert {str(i): v for i, v in r["kept"].items()} == ex["no_abort"]["kept"]
    r = _run(ex, ex["dual"]["m_up"])
    assert {str(i): v for i, v in r["kept"].items()} == ex["dual"]["kept"]
    assert {str(i): v for i, v in r["done_step"].items()} == ex["dual"]["done_step"]
    assert r["steps"] == ex["dual"]["steps"]
    assert r["tokens_decoded"] == ex["dual"]["tokens_decoded"]
    assert r["pages_end"] == 0


def test_appendix_deficit():
    ex = GOLD
    d = ex["deficit"]
    r = _run(ex, 4, draws=d["draws"], mlp=d["mean_lp"], m=d["m"], k=d["k"], cap=d["cap"])
    assert {str(i): v for i, v in r["kept"].items()} == d["kept"]
    assert {str(i): v for i, v in r["done_step"].items()} == d["done_step"]


def _members(rng, m, cap, tie_heavy):
    out = []
    for j in range(m):
        d = int(rng.integers(1, cap + 6))
        trunc = d > cap
        ln = min(d, cap)
        mlp = -float(rng.integers(0, 4 if tie_heavy else 1000)) / 4.0
        out.append(dict(g=100 + j, status=TRUNC if trunc else EOS, length=ln, trunc=trunc,
                        mean_lp=mlp))
    return out


def _brute_short(mem, k):
    """Among all k-subsets, the one whose sorted key vector is lexicographically
    smallest under the shortest-first order: valid beats truncated, shorter
    beats longer, higher mean log-prob beats lower, lower id beats higher."""
    best = None
    for sub in itertools.combinations(mem, k):
        v = sorted(((1 if t["trunc"] else 0), t["length"], -t["mean_lp"] + 0.0, t["g"]) for t in sub)
        if best is None or v < best[0]:
            best = (v, [x[3] for x in v])
    return best[1]


def _brute_dual(mem, k, L):
    """Enumerate (short-set, long-set) pairs: the short set is the best K-subset
    by the shortest-first order; the long set is the best L-subset of the
    remaining valid members by length descending, mean log-prob descending, id."""
    K = k - L
    short = _brute_short(mem, K) if K > 0 else []
    rest = [t for t in mem if t["g"] not in short and not t["trunc"]]
    best = None
    for sub in itertools.combinations(rest, min(L, len(rest))):
        v = sorted((-t["length"], -t["mean_lp"] + 0.0, t["g"]) for t in sub)
        if best is None or v < best[0]:
            best = (v, [x[2] for x in v])
    longs = best[1] if best else []
    chosen = short + longs
    remaining = [t for t in mem if t["g"] not in chosen]
    fill = _brute_short(remaining, k - len(chosen)) if k > len(chosen) else []
    return short + longs + fill


@pytest.mark.parametrize("seed", range(40))
def test_brute_force_short_and_dual(seed):
    rng = np.random.default_rng(seed)
    m = int(rng.integers(2, 9))
    k = int(rng.integers(1, m + 1))
    mem = _members(rng, m, cap=12, tie_heavy=seed % 2 == 0)
    assert select_short(mem, k) == _brute_short(mem, k)
    if k >= 2:
        L = int(rng.integers(1, k))
        assert select_dual(mem, k, L) == _brute_dual(mem, k, L)


def test_nk_special_values():
    assert nk(float("nan")) == float("inf")
    assert nk(-0.0) == 0.0 and str(nk(-0.0)) == "0.0"
    assert nk(0.0) == 0.0 and str(nk(0.0)) == "0.0"
    assert nk(-1.5) == 1.5


@pytest.mark.parametrize("seed", range(12))
def test_early_stop_equals_offline_and_invariants(seed):
    rng = np.random.default_rng(1000 + seed)
    P, m, k, cap, Lp = 6, 8, 4, 40, 16
    draws = np.maximum(1, np.rint(15 * np.exp(0.9 * rng.standard_normal(P * m)))).astype(int)
    mlp = -(np.floor(rng.random(P * m) * 8) / 4).astype(np.float32)   # frequent ties
    es = schedule_only(draws, P, m, k, cap, Lp, mean_lp=mlp, page=4)
    off = schedule_only(draws, P, m, k, cap, Lp, mean_lp=mlp, page=4, early_stop=False)
    assert es["kept"] == off["kept"]
    assert es["pages_end"] == 0 and off["pages_end"] == 0
    assert es["tokens_decoded"] <= off["tokens_decoded"]
    assert es["steps"] <= off["steps"]
    for i in range(P):
        kp = es["kept"][i]
        assert len(kp) == k and len(set(kp)) == k
        assert all(i * m <= g < (i + 1) * m for g in kp)
        assert all(es["length"][g] <= cap for g in kp)
    # processing order: permute which trajectory sits in which slot of its group
    perm = []
    for i in range(P):
        pj = rng.permutation(m)
        perm += [i * m + int(j) for j in pj]
    d2 = draws[perm]
    m2 = mlp[perm]
    # ids change with the permutation; map back and compare as sets of
    # (length, mean_lp) since ids only break exact ties
    r2 = schedule_only(d2, P, m, k, cap, Lp, mean_lp=m2, page=4)
    for i in range(P):
        a = sorted((es["length"][g], float(mlp[g])) for g in es["kept"][i])
        b = sorted((r2["length"][g], float(m2[g])) for g in r2["kept"][i])
        assert a == b
    assert r2["steps"] == es["steps"] and r2["tokens_decoded"] == es["tokens_decoded"]


def test_group_decision_waits_when_not_enough_valid():
    mem = [dict(g=0, status=EOS, length=3, trunc=False, mean_lp=-1.0),
           dict(g=1, status=LIVE, length=3, trunc=False, mean_lp=-1.0),
           dict(g=2, status=LIVE, length=3, trunc=False, mean_lp=-1.0),
           dict(g=3, status=TRUNC, length=3, trunc=True, mean_lp=-1.0)]
    assert group_decision(mem, 2, 1, 4)[0] is False
    mem[1]["status"] = EOS
    c, kept, ab = group_decision(mem, 2, 1, 4)
    assert c and kept == [0, 1] and ab == [2]
    # dual mode waits for every member
    assert group_decision(mem, 2, 1, 5)[0] is False


def test_reclaimed_pages_hand_example_and_conservation():
    from oracle.selection import reclaimed_pages
    # 3 groups of m = 2; groups 0 and 2 complete
    lists = [[5, 6], [], [1], [2], [9, 7, 8], [3]]
    assert reclaimed_pages(lists, {2, 0}, 2) == [5, 6, 9, 7, 8, 3]
    assert reclaimed_pages(lists, set(), 2) == []
    import numpy as np
    rng = np.random.default_rng(1)
    m, n_groups = 4, 50
    sizes = rng.integers(0, 6, n_groups * m)
    perm = rng.permutation(int(sizes.sum()))
    off = np.concatenate([[0], np.cumsum(sizes)])
    lists = [list(perm[off[g]:off[g + 1]]) for g in range(n_groups * m)]
    done = set(int(i) for i in rng.choice(n_groups, 20, replace=False))
    got = reclaimed_pages(lists, done, m)
    want = sorted(p for i in done for j in range(m) for p in lists[i * m + j])
    assert sorted(got) == want and len(set(got)) == len(got)

"""Pins for the oracle sampler: own float32 logarithm vs the library
logarithm, softmax/log-prob/entropy vs brute-force definitions and closed
forms, and the Gumbel-max token distribution vs softmax."""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle.fp32math import ln_f32, gumbel_f32
from oracle.sampler import logprob_entropy, sample_row, sample_token, gumbel_noise
from oracle.philox import philox_words, u24_odd


def _all_u():
    k = np.arange(1 << 23, dtype=np.uint64) * 2 + 1
    return (k.astype(np.float32) * np.float32(2.0 ** -24)).astype(np.float32)


def test_own_ln_close_to_libm_all_u():
    u = _all_u()
    a = ln_f32(u).astype(np.float64)
    ref = np.log(u.astype(np.float64))
    ulp = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)
    assert (np.abs(a - ref) / ulp).max() < 4.0


def test_own_ln_close_to_libm_inner_values():
    x = (-ln_f32(_all_u())).astype(np.float32)
    b = ln_f32(x).astype(np.float64)
    ref = np.log(x.astype(np.float64))
    ulp = np.spacing(np.maximum(np.abs(ref), 1e-38).astype(np.float32)).astype(np.float64)
    assert (np.abs(b - ref) / ulp).max() < 4.0


def test_own_ln_exact_points():
    x = np.array([1.0, 2.0, 0.5, 4.0, 2.0 ** -20], dtype=np.float32)
    got = ln_f32(x).astype(np.float64)
    assert got[0] == 0.0
    for v, g in zip(x[1:], got[1:]):
        assert abs(g - math.log(float(v))) <= 2e-7 * max(1.0, abs(math.log(float(v))))


def test_gumbel_monotone_in_u():
    u = _all_u()[::997]
    g = gumbel_f32(u).astype(np.float64)
    assert (np.diff(g) >= 0).all()       # -ln(-ln u) increases with u


def _brute(z):
    """log-sum-exp, log-probs and entropy with exact rational sums of
    extended-precision exponentials."""
    z = [float(v) for v in z]
    mx = max(z)
    ex = [Fraction(math.exp(v - mx)) for v in z]
    s = sum(ex)
    lse = mx + math.log(float(s))
    p = [float(e / s) for e in ex]
    ent = -sum(pi * math.log(pi) for pi in p if pi > 0)
    return lse, p, ent


@pytest.mark.parametrize("V", [1, 2, 3, 7, 16])
def test_logprob_entropy_brute_force(V):
    rng = np.random.default_rng(V)
    z = rng.normal(0, 3, V)
    lse, p, ent = _brute(z)
    for t in range(V):
        lp, e = logprob_entropy(z, 1.0, t)
        assert abs(lp - (z[t] - lse)) < 1e-12
        assert abs(e - ent) < 1e-12


def test_closed_forms():
    V = 512
    lp, e = logprob_entropy(np.full(V, 0.7), 1.0, 3)
    assert abs(lp + math.log(V)) < 1e-12 and abs(e - math.log(V)) < 1e-12
    a = 1.3
    lp, e = logprob_entropy(np.array([a, 0.0]), 1.0, 0)
    p = 1 / (1 + math.exp(-a))
    assert abs(e - (-p * math.log(p) - (1 - p) * math.log(1 - p))) < 1e-12
    assert abs(lp - math.log(p)) < 1e-12
    z = np.zeros(1000)
    z[5] = 40.0
    lp, e = logprob_entropy(z, 1.0, 5)
    assert e < 1e-12 * 1e3 and abs(lp) < 1e-14 * 1e3
    # temperature scales the logits
    z = np.array([1.0, 2.0, 3.0])
    lp2, e2 = logprob_entropy(z, 2.0, 1)
    lp1, e1 = logprob_entropy(z / 2.0, 1.0, 1)
    assert abs(lp2 - lp1) < 1e-15 and abs(e2 - e1) < 1e-15


def test_masked_logits():
    """Entries at -inf have probability 0: the scores equal those of the
    finite sub-vocabulary (0 log 0 = 0), and the sampled token is never a
    masked one."""
    z = np.full(64, -np.inf)
    z[[3, 17, 40]] = [0.5, 0.5, 0.5]
    lp, e = logprob_entropy(z, 1.0, 17)
    assert abs(e - math.log(3)) < 1e-12 and abs(lp + math.log(3)) < 1e-12
    sub = np.array([1.0, -2.0, 0.25])
    z[[3, 17, 40]] = sub
    lp, e = logprob_entropy(z, 1.0, 40)
    lp_s, e_s = logprob_entropy(sub, 1.0, 2)
    assert abs(lp - lp_s) < 1e-12 and abs(e - e_s) < 1e-12
    for t in range(20):
        assert sample_token(z.astype(np.float32), 1.0, t, 0, 5) in (3, 17, 40)


def test_gumbel_max_frequencies_match_softmax():
    V = 8
    z = np.array([0.3, -1.2, 2.0, 0.0, 1.1, -0.4, 0.8, -2.5])
    p = np.exp(z - z.max())
    p /= p.sum()
    n = 1 << 20
    # counters: trajectory id varies, step fixed
    idx = np.arange(V, dtype=np.uint64)
    traj = np.arange(n, dtype=np.uint64)
    w = philox_words(idx[None, :], traj[:, None], 0, 2, 99)
    g = gumbel_f32(u24_odd(w))
    sc = (z.astype(np.float32)[None, :] + g).astype(np.float32)
    tok = np.argmax(sc, axis=1)
    cnt = np.bincount(tok, minlength=V)
    chi2 = ((cnt - n * p) ** 2 / (n * p)).sum()
    assert chi2 < 30.0     # 7 dof: the 99.99% quantile is about 29.9
    # the vectorised path agrees with the per-row function
    for t in (0, 1, 12345):
        assert sample_token(z.astype(np.float32), 1.0, t, 0, 99) == tok[t]


def test_argmax_ties_lowest_index():
    # identical logits and identical noise cannot happen across indices, but
    # the rule is the numpy first-maximum rule: check it on the score level.
    sc = np.array([1.0, 3.0, 3.0, 2.0], dtype=np.float32)
    assert int(np.argmax(sc)) == 1


def test_sample_row_force_scores_forced_token():
    z = np.array([0.0, 1.0, 2.0, 3.0])
    tok, lp, ent = sample_row(z, 1.0, 5, 3, 7, force=0)
    lp0, ent0 = logprob_entropy(z, 1.0, 0)
    assert lp == lp0 and ent == ent0
    assert tok == sample_token(z.astype(np.float32), 1.0, 5, 3, 7)

"""Gumbel-max sampling with per-token log-probability and entropy.

Definitions (the per-token scoring of the rollout; the paper itself uses its
rollout engine's sampler and states no formula):
    z_i      = logit_i / T                                  (float32 division)
    u_i      = Philox(key=seed, counter=(i>>2, g, s, TAG_SAMPLE)) word i&3 -> (0,1)
    token    = argmax_i fl32(z_i + g(u_i)), smallest i on ties (Gumbel-max)
    logprob  = z_taken - log sum_j exp(z_j)
    entropy  = -sum_i p_i log p_i = LSE(z) - sum_i p_i z_i
``g`` is the trajectory id, ``s`` the 0-based index of the generated token.
The taken token is the forced one when a force is given (forced end of
sequence, or teacher forcing), otherwise the sampled one.

LSE, log-prob and entropy are evaluated in float64 (error far below the
tolerances).  The argmax is made in float32, the kernel's precision.

Pins: brute-force definitions in extended precision on tiny vocabularies,
closed forms (uniform, two-point, one dominant logit), and a chi-square test of
token frequencies against softmax (tests/test_oracle_sampler.py).
"""
import numpy as np

from .philox import philox_words, u24_odd
from .fp32math import gumbel_f32

TAG_SAMPLE = 2


def gumbel_noise(vocab, traj, step, seed):
    idx = np.arange(vocab, dtype=np.uint64)
    return gumbel_f32(u24_odd(philox_words(idx, traj, step, TAG_SAMPLE, seed)))


def perturbed_scores(logits32, temperature, traj, step, seed):
    z = np.asarray(logits32, dtype=np.float32)
    if temperature != 1.0:
        z = (z / np.float32(temperature)).astype(np.float32)
    return (z + gumbel_noise(z.shape[-1], traj, step, seed)).astype(np.float32)


def sample_token(logits32, temperature, traj, step, seed):
    sc = perturbed_scores(logits32, temperature, traj, step, seed)
    return int(np.argmax(sc))     # numpy argmax returns the first maximal index


def top2_margin(logits32, temperature, traj, step, seed):
    sc = np.sort(perturbed_scores(logits32, temperature, traj, step, seed).astype(np.float64))
    return float(sc[-1] - sc[-2]) if sc.size > 1 else float("inf")


def logprob_entropy(logits, temperature, token):
    """log p(token) and entropy of softmax(logits / T), evaluated in float64.
    Logits of -inf (masked entries) have probability 0 and, with the usual
    convention 0 log 0 = 0, contribute nothing to the entropy."""
    z = np.asarray(logits, dtype=np.float64) / float(temperature)
    mx = np.max(z)
    e = np.exp(z - mx)
    ssum = np.sum(e)
    lse = mx + np.log(ssum)
    p = e / ssum
    live = p > 0                                    # 0 log 0 = 0 (masked -inf logits)
    ent = lse - np.sum(p[live] * z[live])
    return float(z[token] - lse), float(ent)


def sample_row(logits, temperature, traj, step, seed, force=-1):
    """Full sampler for one row.  ``logits`` may be float64 (oracle forward) or
    float32 (given inputs); the argmax uses their float32 rounding."""
    l64 = np.asarray(logits, dtype=np.float64)
    tok = sample_token(l64.astype(np.float32), temperature, traj, step, seed)
    taken = tok if force < 0 else int(force)
    lp, ent = logprob_entropy(l64, temperature, taken)
    return tok, lp, ent

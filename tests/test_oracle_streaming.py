"""Pins for the oracle's token-chunk streaming (Sec. 4.3.2): nothing lost or
repeated, dispatch steps follow the threshold rule, one final mark per
trajectory, and threshold 1 is per-step delivery."""
import numpy as np
import pytest

from oracle.streaming import stream_chunks
from oracle.rollout import schedule_only


def _rollout(seed=0, P=5, m=8, k=4, cap=50):
    rng = np.random.default_rng(seed)
    forced = rng.integers(1, 70, P * m)
    s = schedule_only(forced, P, m, k, cap, 16, mean_lp=np.zeros(P * m, np.float32))
    length = {g: s["length"][g] for g in range(P * m)}
    tokens = {g: list(rng.integers(0, 1000, length[g])) for g in length}
    lps = {g: list(-rng.random(length[g])) for g in length}
    status = {g: s["status"][g] for g in length}
    return length, tokens, lps, status, s["steps"]


@pytest.mark.parametrize("threshold", [1, 7, 64, 500, 10 ** 9])
def test_concatenation_and_final_marks(threshold):
    length, tokens, lps, status, steps = _rollout()
    out = stream_chunks(length, tokens, lps, status, steps, threshold)
    got = {g: [] for g in length}
    got_lp = {g: [] for g in length}
    finals = {g: 0 for g in length}
    for step, chunks in out:
        for g, start, tk, lp, fin in chunks:
            assert start == len(got[g])                      # contiguous, in order
            got[g] += tk
            got_lp[g] += lp
            if fin:
                finals[g] += 1
                assert fin == status[g] and len(got[g]) == length[g]
    for g in length:
        assert got[g] == tokens[g] and got_lp[g] == lps[g]
        assert finals[g] == 1
    assert out[-1][0] == steps                                 # final flush


def test_dispatch_steps_follow_the_threshold():
    length, tokens, lps, status, steps = _rollout(seed=3)
    thr = 40
    out = stream_chunks(length, tokens, lps, status, steps, thr)
    # recompute the pending total step by step from the lengths alone
    sent, disp = 0, []
    for s in range(1, steps + 1):
        produced = sum(min(l, s) for l in length.values())
        if produced - sent >= thr:
            disp.append(s)
            sent = produced
    disp_steps = [s for s, _ in out]
    assert disp_steps[:len(disp)] == disp
    assert set(disp_steps) - set(disp) <= {steps}


def test_threshold_one_is_per_step_delivery():
    length, tokens, lps, status, steps = _rollout(seed=5)
    out = stream_chunks(length, tokens, lps, status, steps, 1)
    for s, chunks in out:
        for g, start, tk, lp, fin in chunks:
            assert start == s - 1 and len(tk) <= 1
            if tk:
                assert tk[0] == tokens[g][s - 1]

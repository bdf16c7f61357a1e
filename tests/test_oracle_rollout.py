"""Oracle rollout invariants on the tiny configuration (float64 model)."""
import numpy as np
import pytest

from oracle import model as M
from oracle.rollout import rollout, schedule_only
from oracle.selection import LIVE, EOS, TRUNC, ABORTED
from workload import get_config, rollout_inputs


@pytest.fixture(scope="module")
def tiny_run():
    cfg, run = get_config("tiny")
    W = M.init_weights(cfg)
    prompts, forced = rollout_inputs(cfg, run)
    r = rollout(cfg, W, prompts, forced, run.m, run.k, run.cap, run.sample_seed)
    return cfg, run, W, prompts, forced, r


def test_tiny_rollout_structure(tiny_run):
    cfg, run, W, prompts, forced, r = tiny_run
    P, m, k, cap = run.n_prompts, run.m, run.k, run.cap
    assert sorted(r.kept) == list(range(P))
    for i, kp in r.kept.items():
        assert len(kp) == k and all(i * m <= g < (i + 1) * m for g in kp)
        assert all(r.length[g] <= cap for g in kp)
    assert r.pages_trace[-1][2] == 0
    for g in r.length:
        assert len(r.tokens[g]) == r.length[g]
        if r.status[g] == EOS:
            assert r.tokens[g][-1] == cfg.vocab - 1
            assert r.length[g] == forced[g]
        assert r.status[g] != LIVE
    assert r.tokens_decoded == sum(r.length.values())


def test_tiny_schedule_matches_model_free_accounting(tiny_run):
    cfg, run, W, prompts, forced, r = tiny_run
    mlp = np.array([r.mean_lp32[g] for g in range(run.n_prompts * run.m)], np.float32)
    s = schedule_only(forced, run.n_prompts, run.m, run.k, run.cap, run.prompt_len,
                      mean_lp=mlp)
    assert s["kept"] == r.kept
    assert s["done_step"] == r.done_step
    assert s["steps"] == r.steps
    assert s["tokens_decoded"] == r.tokens_decoded
    assert s["pages_hwm"] == r.pages_hwm
    assert s["pages_end"] == 0


def test_prompt_subset_equals_full_run_slice(tiny_run):
    cfg, run, W, prompts, forced, r = tiny_run
    sub = rollout(cfg, W, prompts, forced, run.m, run.k, run.cap, run.sample_seed, prompt_ids=[2])
    for g in range(2 * run.m, 3 * run.m):
        assert sub.tokens[g] == r.tokens[g]
        assert np.allclose(sub.logprobs[g], r.logprobs[g], atol=1e-12, rtol=0)
    assert sub.kept[2] == r.kept[2] and sub.done_step[2] == r.done_step[2]


def test_logprob_and_entropy_ranges(tiny_run):
    cfg, run, W, prompts, forced, r = tiny_run
    lv = np.log(cfg.vocab)
    for g in r.logprobs:
        assert all(lp <= 0 for lp in r.logprobs[g])
        assert all(0 <= e <= lv + 1e-12 for e in r.entropies[g])


def test_no_abort_counterfactual_same_kept(tiny_run):
    cfg, run, W, prompts, forced, r = tiny_run
    mlp = np.array([r.mean_lp32[g] for g in range(run.n_prompts * run.m)], np.float32)
    s = schedule_only(forced, run.n_prompts, run.m, run.k, run.cap, run.prompt_len,
                      mean_lp=mlp, early_stop=False)
    assert s["kept"] == r.kept
    assert s["steps"] >= r.steps and s["tokens_decoded"] >= r.tokens_decoded


# ---------------------------------------------------------------- ragged plans
def _ragged_plan(P, k, m):
    """A redundancy plan with sizes in [k, m]: shortest-only and dual-end groups mixed."""
    return [m if i % 2 == 0 else k + (i % (m - k + 1)) for i in range(P)]


def test_ragged_schedule_equals_per_prompt_uniform_runs():
    """A batch with per-prompt candidate counts decides every group exactly as a
    batch holding only that prompt with a uniform size M'_i would (groups are
    independent; pages are additive)."""
    rng = np.random.default_rng(8)
    P, m, k, cap, Lp = 6, 8, 4, 40, 32
    forced = rng.integers(1, 60, P * m)
    mlp = -(np.floor(rng.random(P * m) * 64) / 64).astype(np.float32)
    plan = _ragged_plan(P, k, m)
    r = schedule_only(forced, P, m, k, cap, Lp, mean_lp=mlp, alloc=plan)
    tok = 0
    for i in range(P):
        mi = plan[i]
        f = forced[i * m:i * m + mi]
        s = schedule_only(f, 1, mi, k, cap, Lp, m_up=2 * k, mean_lp=mlp[i * m:i * m + mi])
        assert r["kept"][i] == [i * m + g for g in s["kept"][0]]
        assert r["done_step"][i] == s["done_step"][0]
        assert r["length"][i * m:i * m + mi] == s["length"]
        assert all(x == 0 for x in r["length"][i * m + mi:(i + 1) * m])
        tok += s["tokens_decoded"]
    assert r["tokens_decoded"] == tok
    assert r["steps"] == max(r["done_step"].values())
    assert r["pages_end"] == 0
    # the uniform plan is the plain batch
    u = schedule_only(forced, P, m, k, cap, Lp, mean_lp=mlp, alloc=[m] * P)
    v = schedule_only(forced, P, m, k, cap, Lp, mean_lp=mlp)
    assert u == v


def test_ragged_model_rollout_matches_schedule(tiny_run):
    cfg, run, W, prompts, forced, r = tiny_run
    plan = _ragged_plan(run.n_prompts, run.k, run.m)
    rr = rollout(cfg, W, prompts, forced, run.m, run.k, run.cap, run.sample_seed, alloc=plan)
    assert sorted(rr.tokens) == [i * run.m + j for i in range(run.n_prompts) for j in range(plan[i])]
    n = run.n_prompts * run.m
    mlp = np.array([rr.mean_lp32.get(g, 0.0) for g in range(n)], np.float32)
    s = schedule_only(forced, run.n_prompts, run.m, run.k, run.cap, run.prompt_len, mean_lp=mlp,
                      alloc=plan)
    assert s["kept"] == rr.kept and s["done_step"] == rr.done_step
    assert s["steps"] == rr.steps and s["tokens_decoded"] == rr.tokens_decoded
    assert s["pages_hwm"] == rr.pages_hwm
    # a trajectory's tokens do not depend on the plan (counter-based sampling)
    for g in rr.tokens:
        L = min(len(rr.tokens[g]), len(r.tokens[g]))
        assert rr.tokens[g][:L] == r.tokens[g][:L]

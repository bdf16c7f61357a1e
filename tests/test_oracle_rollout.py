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

"""The seeded input generators: the sizing the configurations are quoted on,
and the per-prompt-spread lengths used to exercise the adaptive allocation."""
import numpy as np

from oracle.rollout import schedule_only
from workload import get_config, rollout_inputs
from workload.gen import heterogeneous_forced_lengths


def test_configuration_schedules():
    """The forced lengths give the schedules the configurations are sized on."""
    for name, steps, tokens in [("tiny", 45, 794), ("dense-small", 1486, 334472),
                                ("qwen3-8b", 2557, 502171), ("qwen3-30b-a3b", 2234, 791511)]:
        model, run = get_config(name)
        _, forced = rollout_inputs(model, run)
        s = schedule_only(forced, run.n_prompts, run.m, run.k, run.cap, run.prompt_len)
        assert (s["steps"], s["tokens_decoded"]) == (steps, tokens), name


def test_heterogeneous_lengths_spread_belongs_to_the_prompt():
    _, run = get_config("qwen3-8b")
    d = heterogeneous_forced_lengths(run, 7).astype(np.float64).reshape(run.n_prompts, run.m)
    ls = np.log(d)
    narrow, wide = ls[0::2].std(axis=1), ls[1::2].std(axis=1)
    assert narrow.mean() < 0.45 < wide.mean()
    # the 5-10x median tail only on the wide prompts
    assert d[0::2].max() < 5 * run.len_median
    assert np.array_equal(heterogeneous_forced_lengths(run, 7), heterogeneous_forced_lengths(run, 7))

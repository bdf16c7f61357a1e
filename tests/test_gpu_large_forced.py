"""Full-depth parity at the two large configurations (Qwen3-8B-shaped dense,
36 layers; Qwen3-30B-A3B-shaped MoE, 48 layers), in the launch configuration
the benchmark times: the whole batch (32 x 16 or 64 x 16 trajectories, every
prompt prefilled) decodes on the GPU while prompts 0 and 1 and their 32
trajectories are teacher-forced with a seeded token table for their first 64
generated tokens.  The expected values come from the layer-major float64
oracle (tests/golden/make_forced_golden.py, oracle/ only).

Compared on every generated token of the subset:
  * logits at 256 fixed vocabulary ids, the row's largest logit and its
    log-sum-exp, within 2e-2 of the row's largest |logit|;
  * log-prob and entropy, the worst deviations printed and bounded by what
    the logit tolerance implies;
  * the GPU's own Gumbel-max sample: bit-exact against the oracle sampler
    run on the GPU's own float32 logits (selected steps), and equal to the
    oracle's sample wherever the oracle's top-2 perturbed-score margin
    exceeds twice the logit tolerance (the only way the argmax can change).
MoE routing is teacher-forced too (darts_debug_moe_routing): every row
combines the oracle's experts, so every row's logits are compared.  The
router's own top-k is checked against the oracle's wherever the oracle's
k / k+1 probability margin exceeds twice the largest router-probability
deviation measured in the same run, and that deviation is bounded."""
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from forced_parity import check_forced, run_forced
from workload import get_config, rollout_inputs

pytestmark = pytest.mark.gpu
GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(config):
    path = os.path.join(GOLD, f"forced_{config}.npz")
    assert os.path.exists(path), f"missing {path}: run tests/golden/make_forced_golden.py {config}"
    return dict(np.load(path))


def _check(config):
    g = _golden(config)
    model, run = get_config(config)
    prompts, forced = rollout_inputs(model, run)
    rec, strict, route = run_forced(model, run, prompts, forced, g, config)
    n = check_forced(model, run, g, rec, strict, route, config)
    # every generated token of the window is compared (no trajectory of prompts
    # 0 and 1 ends or is aborted inside it at these lengths)
    assert n == int(g["n_gen"].sum()), (n, int(g["n_gen"].sum()))


def test_qwen3_8b_full_depth_teacher_forced():
    _check("qwen3-8b")


def test_qwen3_30b_a3b_full_depth_teacher_forced():
    _check("qwen3-30b-a3b")

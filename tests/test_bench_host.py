"""Host-side parts of bench.py: the CPU baseline runs the oracle on dense and
mixture-of-experts shapes and reports a rate and the threads it used; the
wall-budget arithmetic never times fewer than one rollout."""
from dataclasses import replace

import pytest

import bench
from workload import get_config


@pytest.mark.parametrize("name", ["dense-small", "qwen3-30b-a3b"])
def test_cpu_baseline_runs_on_shrunk_configs(name):
    model, run = get_config(name)
    # same structure (dense SwiGLU or routed experts), shrunk to seconds of CPU work
    model = replace(model, n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=2, head_dim=64, vocab=512,
                    ffn_dim=0 if model.is_moe else 512, expert_ffn=256 if model.is_moe else 0,
                    n_experts=16 if model.is_moe else 0, top_k=4 if model.is_moe else 0)
    run = replace(run, prompt_len=64, m=4, k=2)
    out = bench.cpu_baseline(model, run, budget_s=0.5)
    assert out["kind"] == "oracle" and out["unit"] == "tokens/s"
    assert out["value"] > 0 and out["cores"] >= 1
    assert isinstance(out["sample"], str) and out["sample"]

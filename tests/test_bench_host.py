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


def test_gap_summary_splits_step_boundaries(tmp_path):
    """Idle time of the last rollout of a kernel trace: a gap after a
    prune_kernel is a step boundary, every other gap is inside a step;
    overlapping kernels count once toward busy time."""
    import csv
    rows = [("init_weights_kernel", 0, 10),
            ("prefill_pages_kernel", 100, 110), ("embed_kernel", 115, 120), ("prune_kernel", 120, 130),
            ("embed_norm_kernel", 180, 200), ("gemm_a", 205, 300), ("gemm_b", 250, 280),
            ("prune_kernel", 300, 310), ("copyBuffer", 320, 325), ("embed_norm_kernel", 400, 410),
            ("prune_kernel", 410, 420)]
    p = tmp_path / "kernel_trace.csv"
    with open(p, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        for n, s, e in rows:
            w.writerow([n, s, e])
    out = bench.summarize_gaps(str(p))
    # boundaries: 130..180 and 310..320..325..400 (a copy after the selection)
    assert out["kernels"] == 10 and out["prune_launches"] == 3
    assert out["step_boundary_idle_s"] == pytest.approx(135e-9)
    assert out["intra_step_idle_s"] == pytest.approx(10e-9)
    assert out["span_s"] == pytest.approx(320e-9) and out["busy_s"] == pytest.approx(175e-9)
    assert out["idle_s"] == pytest.approx(145e-9)


def test_pmc_class_reads_the_epilogue_argument():
    import bench
    assert bench._pmc_class("void darts::attn_bf16_db_kernel<128>(darts::AttnBf16Args)") == "attention"
    gu = "void darts::gemm_dma_grouped_kernel<96, 128, 64, 2, 2, 3, 3, true>(unsigned short const*, int)"
    dn = "void darts::gemm_dma_grouped_kernel<64, 128, 64, 2, 2, 3, 1, false>(unsigned short const*, int)"
    assert bench._pmc_class(gu) == "expert_gate_up"
    assert bench._pmc_class(dn) == "expert_down"
    assert bench._pmc_class("void darts::gemm_dma_kernel<128, 128, 64, 2, 2, 4, 3, false>(int)") is None
    assert bench._pmc_class("void darts::gemm_wd_grouped_kernel<96, 32, 2, 3>(unsigned short const*)") == \
        "expert_gate_up"

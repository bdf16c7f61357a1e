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


def _write_counters(path, rows):
    """A rocprofv3 --pmc counter_collection.csv: (dispatch id, kernel, counter, value) rows;
    a dispatch may have several rows (one per hardware block), which are summed."""
    import csv
    path.mkdir(parents=True, exist_ok=True)
    with open(path / "run_counter_collection.csv", "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for r in rows:
            w.writerow(r)


def test_pmc_summary_scales_by_the_copy_calibration(tmp_path):
    """Per-launch traffic = mean counter KiB per dispatch x 1024 x (1 GiB / what
    the counter reads for a 1 GiB copy), per kernel class; unrelated kernels
    are ignored; the expert classes carry the expert-GEMM source hash."""
    import json
    # FETCH_SIZE reads half of a copy's bytes (scale 2), WRITE_SIZE all of them (scale 1)
    _write_counters(tmp_path / "pmc_copy_FETCH_SIZE",
                    [(i, "copyBuffer", "FETCH_SIZE", 524288.0) for i in range(3)])
    _write_counters(tmp_path / "pmc_copy_WRITE_SIZE",
                    [(i, "copyBuffer", "WRITE_SIZE", 1048576.0) for i in range(3)])
    attn = "void darts::attn_bf16_db_kernel<128>(darts::AttnBf16Args)"
    gu = "void darts::gemm_wd_grouped_kernel<64, 32, 2, 3>(unsigned short const*)"
    dn = "void darts::gemm_dma_grouped_kernel<64, 128, 64, 2, 2, 3, 1, false, 2>(unsigned short const*)"
    _write_counters(tmp_path / "pmc_moe_FETCH_SIZE",
                    [(1, attn, "FETCH_SIZE", 600.0), (1, attn, "FETCH_SIZE", 400.0),   # one dispatch, two rows
                     (2, attn, "FETCH_SIZE", 3000.0), (3, gu, "FETCH_SIZE", 5000.0),
                     (4, dn, "FETCH_SIZE", 2500.0), (5, "void darts::other_kernel()", "FETCH_SIZE", 9e9)])
    _write_counters(tmp_path / "pmc_moe_WRITE_SIZE",
                    [(1, attn, "WRITE_SIZE", 10.0), (2, attn, "WRITE_SIZE", 30.0),
                     (3, gu, "WRITE_SIZE", 100.0), (4, dn, "WRITE_SIZE", 200.0)])
    line = {"config": {"workload": "synthetic"},
            "roofline": {"algorithmic_bytes_per_launch": 4096.0 * 1024},
            "roofline_moe_experts": {"expert_gate_up": {"algorithmic_bytes_per_launch": 10240.0 * 1024},
                                     "expert_down": {"algorithmic_bytes_per_launch": 5000.0 * 1024}}}
    (tmp_path / "bench_moe.json").write_text("[bench] log line\n" + json.dumps(line) + "\n")
    out = bench.summarize_pmc(str(tmp_path), name="moe")
    cal = out["copy_calibration"]
    assert cal["FETCH_SIZE"]["scale"] == pytest.approx(2.0) and cal["WRITE_SIZE"]["scale"] == pytest.approx(1.0)
    k = out["kernels"]
    assert set(k) == {"attention", "expert_gate_up", "expert_down"}
    a = k["attention"]
    assert a["launches_FETCH_SIZE"] == 2 and a["launches_WRITE_SIZE"] == 2
    assert a["fetch_bytes_per_launch"] == pytest.approx((1000.0 + 3000.0) / 2 * 1024 * 2)
    assert a["write_bytes_per_launch"] == pytest.approx(20.0 * 1024)
    assert a["measured_over_algorithmic"] == pytest.approx((4000.0 + 20.0) / 4096.0)
    assert out["traffic_bytes_per_launch"] == pytest.approx(a["traffic_bytes_per_launch"])
    assert k["expert_gate_up"]["traffic_bytes_per_launch"] == pytest.approx((10000.0 + 100.0) * 1024)
    assert k["expert_down"]["measured_over_algorithmic"] == pytest.approx((5000.0 + 200.0) / 5000.0)
    assert out["kernel_source_sha256"] == bench.attn_source_hash()
    assert k["expert_down"]["kernel_source_sha256"] == bench.source_hash(bench.EXPERT_SOURCES)
    assert out["workload"] == "synthetic"


def test_mfma_summary_weights_dispatches_by_active_cycles(tmp_path):
    """MFMA busy of a kernel = sum(active cycles x MfmaUtil%) / sum(active cycles)
    over its dispatches; the argument list is dropped from the kernel name."""
    k1 = "void darts::gemm_dma_kernel<128, 128, 64, 2, 2, 4, 0, false>(unsigned short const*, int)"
    k2 = "void darts::gemm_wd_grouped_kernel<64, 32, 2, 3>(unsigned short const*)"
    rows = []
    for did, name, gui, util, flop in ((1, k1, 100.0, 50.0, 1e9), (2, k1, 300.0, 10.0, 2e9),
                                       (3, k2, 1000.0, 20.0, 5e9)):
        rows += [(did, name, "GRBM_GUI_ACTIVE", gui), (did, name, "MfmaUtil", util),
                 (did, name, "MfmaFlopsBF16", flop)]
    _write_counters(tmp_path / "mf", rows)
    out = bench.summarize_mfma(str(tmp_path / "mf"))
    a = out["kernels"]["gemm_dma_kernel<128, 128, 64, 2, 2, 4, 0, false>"]
    assert a["dispatches"] == 2 and a["active_cycles"] == pytest.approx(400.0)
    assert a["mfma_util"] == pytest.approx((100 * 0.5 + 300 * 0.1) / 400)
    assert a["bf16_flop"] == pytest.approx(3e9)
    t = out["all_gemm_kernels"]
    assert t["dispatches"] == 3
    assert t["mfma_util"] == pytest.approx((50 + 30 + 200) / 1400)
    assert list(out["kernels"])[0] == "gemm_wd_grouped_kernel<64, 32, 2, 3>"   # most active first

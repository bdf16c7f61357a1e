#!/usr/bin/env python3
"""Rollout benchmark on one MI355X.

A step is one whole rollout of one batch through the C ABI: darts_reset,
darts_prefill, then darts_decode_step + darts_select_and_prune until every
prompt's kept set is complete (proactive early stopping, KV page reclaim).
Inputs (weights, prompts, forced lengths) are resident in HBM before timing.

Prints ONE JSON line: rollout tokens/s (all generated tokens, including the
ones of trajectories later aborted) over the timed steps, time-to-kept-set,
the decode-attention roofline (HBM), GEMM MFMA utilisation, and the CPU
oracle timed on a bounded sample of the same workload.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3       # fp32 vector / MFMA


def workload_desc(model, run):
    tail = " +5% tail at 5-10x median" if run.len_tail else ""
    return (f"{model.name} rollout: {model.n_layers} layers, d {model.d_model}, "
            f"{model.n_q_heads}/{model.n_kv_heads} heads x {model.head_dim}, "
            f"{'MoE %d experts top-%d' % (model.n_experts, model.top_k) if model.n_experts else 'FFN %d' % model.ffn_dim}, "
            f"vocab {model.vocab}; {run.n_prompts} prompts x {run.prompt_len} tokens, m={run.m}, k={run.k}, "
            f"cap {run.cap}, forced lengths lognormal(median {run.len_median:g}, sigma {run.len_sigma:g}){tail}")


def cpu_baseline(model, run, budget_s=20.0):
    """The oracle's decode step (float64 numpy forward + Gumbel-max sampler) on
    one prompt group (m rows) at context prompt_len + 512, timed per layer and
    for the fixed part (embedding, final norm, LM head, sampler), scaled to the
    model's layer count.  Weights are constant-filled matrices of the real
    shapes: dense float64 products cost the same for any values, and
    generating the Philox weights would only add setup time."""
    import numpy as np
    from oracle import model as OM
    from oracle.sampler import sample_row
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    rng = np.random.default_rng(0)
    d, hq, hkv, hd, F, V = (model.d_model, model.n_q_heads, model.n_kv_heads, model.head_dim,
                            model.ffn_dim, model.vocab)

    def layer():
        r = lambda *s: np.full(s, 1.0 / s[-1])
        return OM.LayerW(wq=r(hq * hd, d), wk=r(hkv * hd, d), wv=r(hkv * hd, d), wo=r(d, hq * hd),
                         wgate=r(F, d), wup=r(F, d), wdown=r(d, F))

    B = run.m
    ctx0 = run.prompt_len + 512
    emb = np.full((V, d), 0.5)
    head = np.full((V, d), 1.0 / d)
    l1, l2 = layer(), layer()
    caches = [(rng.standard_normal((B, ctx0, hkv, hd)), rng.standard_normal((B, ctx0, hkv, hd)))
              for _ in range(2)]
    toks = rng.integers(0, V, B)
    W1 = OM.Weights(embed=emb, layers=[l1], lm_head=head)
    W2 = OM.Weights(embed=emb, layers=[l1, l2], lm_head=head)
    t_one, t_two, t_samp = [], [], []
    t_start = time.perf_counter()
    reps = 0
    while True:
        t0 = time.perf_counter()
        lg, _ = OM.decode_batch(model, W1, toks, caches[:1])
        t1 = time.perf_counter()
        OM.decode_batch(model, W2, toks, caches)
        t2 = time.perf_counter()
        for b in range(B):
            sample_row(lg[b], 1.0, b, 0, 1)
        t3 = time.perf_counter()
        t_one.append(t1 - t0)
        t_two.append(t2 - t1)
        t_samp.append(t3 - t2)
        reps += 1
        if time.perf_counter() - t_start > budget_s or reps >= 20:
            break
    one, two, samp = (float(np.median(t_one)), float(np.median(t_two)), float(np.median(t_samp)))
    per_layer = max(two - one, 1e-9)
    fixed = max(one - per_layer, 0.0) + samp
    step_s = fixed + model.n_layers * per_layer
    return {"value": B / step_s, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": (f"oracle float64 decode step of one prompt group ({B} rows) at context {ctx0}: "
                       f"1- and 2-layer forwards (per layer {per_layer:.3f} s, fixed part incl. "
                       f"LM head and {B} Gumbel-max samples {fixed:.3f} s) scaled to "
                       f"{model.n_layers} layers; {reps} repetitions, "
                       f"{time.perf_counter() - t_start:.1f} s of CPU work")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="qwen3-8b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-abort", action="store_true", help="counterfactual without early stop")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: this build runs the rollout of one data-parallel "
              "rank (prompt groups are independent); multi-GPU runs are not part of it.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2605_30859_amd import binding as B
    from workload import get_config, rollout_inputs

    torch.cuda.set_device(0)
    B.load_library()
    model, run = get_config(args.config)
    prompts, forced = rollout_inputs(model, run)
    flags = B.FLAG_TIMING | (B.FLAG_NO_ABORT if args.no_abort else 0)
    t_init = time.perf_counter()
    ro = B.Rollout(model, run, flags=flags)
    pr = torch.from_numpy(prompts.reshape(-1).copy()).cuda()
    fl = torch.from_numpy(forced.astype(np.int32)).cuda()
    torch.cuda.synchronize()
    t_init = time.perf_counter() - t_init
    print(f"[bench] {args.config}: context ready in {t_init:.1f} s", file=sys.stderr, flush=True)

    def one_rollout():
        ro.darts_reset()
        t0 = time.perf_counter()
        ro.darts_prefill(pr, fl)
        ro.darts_select_and_prune()
        steps = 1
        while ro.n_done < run.n_prompts:
            ro.darts_decode_step()
            ro.darts_select_and_prune()
            steps += 1
            if steps % 200 == 0:
                print(f"[bench]   step {steps}: live {ro.n_live}, done {ro.n_done}",
                      file=sys.stderr, flush=True)
        torch.cuda.synchronize()
        return time.perf_counter() - t0, ro.stats()

    for w in range(args.warmup):
        dt, st = one_rollout()
        print(f"[bench] warmup {w}: {dt:.2f} s, {st['tokens_decoded']} tokens", file=sys.stderr,
              flush=True)
    torch.cuda.synchronize()
    walls, stats = [], []
    t0 = time.perf_counter()
    for k in range(args.steps):
        dt, st = one_rollout()
        walls.append(dt)
        stats.append(st)
        print(f"[bench] step {k}: {dt:.2f} s, {st['tokens_decoded']} tokens, "
              f"{st['steps']} sampling steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    total = time.perf_counter() - t0
    tokens = sum(s["tokens_decoded"] for s in stats)
    attn_ms = sum(s["attn_ms"] for s in stats)
    attn_b = sum(s["attn_bytes"] for s in stats)
    attn_n = sum(s["attn_launches"] for s in stats)
    gemm_ms = sum(s["gemm_ms"] for s in stats)
    gemm_f = sum(s["gemm_flop"] for s in stats)
    ach = attn_b / (attn_ms * 1e-3) / 1e9 if attn_ms > 0 else 0.0
    peak_mm = BF16_PEAK_TFLOPS if model.dtype == "bf16" else FP32_PEAK_TFLOPS
    gemm_tf = gemm_f / (gemm_ms * 1e-3) / 1e12 if gemm_ms > 0 else 0.0
    cls = {}
    for i, name in enumerate(["qkv", "o", "gate_up", "down", "lm_head"]):
        ms = sum(s["gemm_cls_ms"][i] for s in stats)
        fl = sum(s["gemm_cls_flop"][i] for s in stats)
        cls[name] = {"ms": ms, "tflops": fl / (ms * 1e-3) / 1e12 if ms > 0 else 0.0}
    ro.close()

    out = {
        "metric": "rollout tokens/s + time-to-kept-set-complete; decode-attn HBM % of peak",
        "value": tokens / total,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * total / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": model.dtype,
        "data": "synthetic (seeded uniform prompt tokens, lognormal forced lengths, Philox random-init weights)",
        "config": {"workload": workload_desc(model, run), "name": args.config,
                   "prompts": run.n_prompts, "m": run.m, "k": run.k, "cap": run.cap,
                   "early_stop": not args.no_abort},
        "time_to_kept_set_s": float(np.mean(walls)),
        "tokens_per_rollout": stats[-1]["tokens_decoded"],
        "sampling_steps": stats[-1]["steps"],
        "pages_hwm": stats[-1]["pages_hwm"],
        "kv_pool_pages": stats[-1]["n_pages"],
        "roofline": {"bound": "hbm", "kernel": "attn_bf16_kernel (paged GQA decode attention)",
                     "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": ach / HBM_PEAK_GBS, "traffic": None,
                     "launches": attn_n, "avg_launch_us": 1e3 * attn_ms / max(attn_n, 1),
                     "algorithmic_bytes_per_launch": attn_b / max(attn_n, 1),
                     "share_of_step_time": attn_ms * 1e-3 / total},
        "gemm": {"bound": "mfma", "achieved": gemm_tf, "peak": peak_mm, "unit": "TFLOP/s",
                 "frac": gemm_tf / peak_mm, "share_of_step_time": gemm_ms * 1e-3 / total,
                 "by_class": cls},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        try:
            out["cpu_baseline"] = cpu_baseline(model, run)
        except Exception as e:  # the baseline is context, never the product path
            out["cpu_baseline"] = {"error": repr(e)}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

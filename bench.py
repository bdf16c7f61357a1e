#!/usr/bin/env python3
"""Rollout benchmark on one MI355X.

A step is one whole rollout of one batch through the C ABI: darts_reset,
darts_prefill, then darts_decode_step + darts_select_and_prune until every
prompt's kept set is complete (proactive early stopping, KV page reclaim).
Inputs (weights, prompts, forced lengths) are resident in HBM before timing.

Prints ONE JSON line: rollout tokens/s (all generated tokens, including the
ones of trajectories later aborted) over the timed steps, time-to-kept-set,
the decode-attention roofline (HBM), GEMM MFMA utilisation, and the CPU
oracle timed on a bounded sample of the same workload.  Kernel durations come
from HIP events the library records around each attention and GEMM launch of
the prefill and of every 8th decode step (totals are scaled to the whole run).
"""
import argparse
import json
import math
import os
import sys
import time

T_PROCESS = time.perf_counter()
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


SUBSET_PROMPTS, SUBSET_STEPS = 2, 64


def cpu_baseline(model, run, budget_s=20.0):
    """The oracle on a bounded sample of the teacher-forced parity subset: two
    prompts and their 2*m trajectories, the whole prompt prefill and the first
    64 generated tokens of each (2*m*64 tokens), as oracle/forced.py computes
    it layer by layer.  Timed: one decoder layer over all the subset's rows
    (scaled by the layer count), the LM head on a sample of rows and the
    Gumbel-max sampler on a sample of rows (scaled to all of them).  Weight
    generation is setup, not timed; the weights are random matrices of the
    real shapes (float64 products cost the same for any values; the router
    is random so that tokens spread over the experts as they would)."""
    import numpy as np
    from dataclasses import replace
    from oracle import model as OM
    from oracle.forced import forced_forward
    from oracle.sampler import sample_row
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    rng = np.random.default_rng(0)
    d, hq, hkv, hd, F, V = (model.d_model, model.n_q_heads, model.n_kv_heads, model.head_dim,
                            model.ffn_dim, model.vocab)
    r = lambda *sh: np.full(sh, 1.0 / sh[-1])
    lw = OM.LayerW(wq=r(hq * hd, d), wk=r(hkv * hd, d), wv=r(hkv * hd, d), wo=r(d, hq * hd))
    if model.is_moe:
        E, Fe = model.n_experts, model.expert_ffn
        lw.router = rng.standard_normal((E, d)) / math.sqrt(d)
        lw.egate, lw.eup, lw.edown = r(E, Fe, d), r(E, Fe, d), r(E, d, Fe)
    else:
        lw.wgate, lw.wup, lw.wdown = r(F, d), r(F, d), r(d, F)
    Ps, m, S, Lp = SUBSET_PROMPTS, run.m, SUBSET_STEPS, run.prompt_len
    T = Ps * m
    prompts = rng.integers(0, V - 1, (Ps, Lp))
    consumed = rng.integers(0, V - 1, (T, S - 1))
    emb = np.full((V, d), 0.5)
    one = replace(model, n_layers=1)
    t_start = time.perf_counter()
    t_layer = []
    while not t_layer or (time.perf_counter() - t_start < 0.5 * budget_s and len(t_layer) < 3):
        t0 = time.perf_counter()
        h_last, h_dec = forced_forward(one, prompts, np.repeat(np.arange(Ps), m), consumed, lambda l: lw,
                                       lambda tk: emb[np.asarray(tk)])
        t_layer.append(time.perf_counter() - t0)
    n_head = min(T * S, 256)
    head = np.full((V, d), 1.0 / d)
    t0 = time.perf_counter()
    lg = h_dec.reshape(-1, d)[:n_head] @ head.T
    t_head = (time.perf_counter() - t0) * (T * S) / n_head
    del head
    n_samp = 0
    t0 = time.perf_counter()
    while n_samp < 4 or (n_samp < n_head and time.perf_counter() - t0 < 0.2 * budget_s):
        sample_row(lg[n_samp], 1.0, n_samp, 0, 1)
        n_samp += 1
    t_samp = (time.perf_counter() - t0) * (T * S) / n_samp
    layer = float(np.median(t_layer))
    total = model.n_layers * layer + t_head + t_samp
    return {"value": T * S / total, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": (f"oracle float64 teacher-forced subset ({Ps} prompts x {Lp} tokens prefilled, "
                       f"{T} trajectories x {S} generated tokens = {T * S} tokens): one decoder layer over "
                       f"all {Ps * Lp + T * (S - 1)} rows {layer:.2f} s (median of {len(t_layer)}) x "
                       f"{model.n_layers} layers, LM head {t_head:.2f} s (timed on {n_head} rows), "
                       f"sampler {t_samp:.2f} s (timed on {n_samp} rows); estimated subset time "
                       f"{total:.1f} s from {time.perf_counter() - t_start:.1f} s of CPU work"),
            "subset_tokens": T * S, "subset_s_estimated": total}


def gpu_subset_rate(B, model, run, reps=2):
    """The GPU on the same subset as cpu_baseline, as a separate small run: a
    batch of the subset's two prompts (their trajectories' lengths capped at
    64 generated tokens, so every one generates exactly 64), prefill plus
    decode steps through the C ABI.  Best of ``reps`` timed runs after one
    untimed run."""
    import numpy as np
    import torch
    from dataclasses import replace
    from workload import rollout_inputs
    sub = replace(run, n_prompts=SUBSET_PROMPTS, cap=SUBSET_STEPS, kv_pool_gb=0.0)
    prompts, _ = rollout_inputs(model, run)
    pr = torch.from_numpy(np.ascontiguousarray(prompts[:SUBSET_PROMPTS].reshape(-1))).cuda()
    fl = torch.full((SUBSET_PROMPTS * run.m,), SUBSET_STEPS + 1, dtype=torch.int32, device="cuda")
    ro = B.Rollout(model, sub, flags=B.FLAG_NO_ABORT)
    best, tokens = float("inf"), 0
    for i in range(reps + 1):
        ro.darts_reset()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ro.darts_prefill(pr, fl)
        ro.darts_select_and_prune()
        while ro.n_done < SUBSET_PROMPTS:
            ro.darts_decode_step()
            ro.darts_select_and_prune()
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        tokens = ro.stats()["tokens_decoded"]
        if i > 0:
            best = min(best, dt)
    ro.close()
    return {"value": tokens / best, "unit": "tokens/s", "tokens": int(tokens), "seconds": best}


def rollout_bound(model, run, rows, hbm_gbs, mfma_tflops):
    """Roofline bound of the measured schedule: per decode step with B live
    rows at context Lp + i, KV bytes / HBM + max(weight bytes / HBM, GEMM
    FLOP / MFMA peak); the prefill adds the prompt tokens' GEMM FLOP (or its
    weight read).  MoE weights count every expert (an upper bound on the
    bytes, so the bound is optimistic there)."""
    d, hq, hkv, hd, L = model.d_model, model.n_q_heads, model.n_kv_heads, model.head_dim, model.n_layers
    eb = 2 if model.dtype == "bf16" else 4
    attn_p = d * (hq + 2 * hkv) * hd + hq * hd * d
    if model.is_moe:
        ffn_all = model.n_experts * 3 * d * model.expert_ffn + d * model.n_experts
        ffn_act = model.top_k * 3 * d * model.expert_ffn + d * model.n_experts
    else:
        ffn_all = ffn_act = 3 * d * model.ffn_dim
    w_bytes = (L * (attn_p + ffn_all) + d * model.vocab) * eb
    flop_tok = 2.0 * (L * (attn_p + ffn_act) + d * model.vocab)
    kv_tok = 2 * L * hkv * hd * eb
    hbm, mm = hbm_gbs * 1e9, mfma_tflops * 1e12
    t = max(w_bytes / hbm, run.n_prompts * run.prompt_len * flop_tok / mm)
    for i, b in enumerate(rows, start=1):
        b = float(b)
        t += b * (run.prompt_len + i) * kv_tok / hbm + max(w_bytes / hbm, b * flop_tok / mm)
    return t


def gemm_class_roofline(model, run, rows, hbm_gbs, mfma_tflops):
    """Per dense GEMM class, the roofline time of the measured schedule in ms:
    every launch costs max(2 M N K / MFMA peak, N K weight bytes / HBM), with
    M = the live rows of each decode step (one launch per layer; the LM head
    once per step) and the prefill's rows.  MoE expert GEMMs are not included."""
    d, hq, hkv, hd, L = model.d_model, model.n_q_heads, model.n_kv_heads, model.head_dim, model.n_layers
    eb = 2 if model.dtype == "bf16" else 4
    shapes = {"qkv": ((hq + 2 * hkv) * hd, d), "o": (d, hq * hd), "lm_head": (model.vocab, d)}
    if not model.is_moe:
        shapes["gate_up"] = (2 * model.ffn_dim, d)
        shapes["down"] = (d, model.ffn_dim)
    hbm, mm = hbm_gbs * 1e9, mfma_tflops * 1e12
    out = {}
    for name, (N, K) in shapes.items():
        per_step = 1 if name == "lm_head" else L
        pre_m = run.n_prompts if name == "lm_head" else run.n_prompts * run.prompt_len
        t = per_step * max(2.0 * pre_m * N * K / mm, N * K * eb / hbm)
        for b in rows:
            t += per_step * max(2.0 * float(b) * N * K / mm, N * K * eb / hbm)
        out[name] = 1e3 * t
    return out


def hbm_read_rate(B, gib=8, reps=10):
    """HBM read rate this device sustains (GB/s): the library's streaming-read
    kernel (16-byte non-temporal loads, 2048 blocks, grid-stride) over a `gib` GiB buffer."""
    import torch
    src = torch.zeros(gib << 30, dtype=torch.uint8, device="cuda")
    sink = torch.empty(8192, dtype=torch.float32, device="cuda")
    for _ in range(2):
        B.darts_stream_read(src, sink)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        B.darts_stream_read(src, sink)
    e1.record()
    torch.cuda.synchronize()
    rate = src.numel() * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, sink
    torch.cuda.empty_cache()
    return rate


def gemm_compare(B, reps=12):
    """The library's bf16 GEMM (its own plan, fp32 output, split-K reduce
    included) against torch.nn.functional.linear (hipBLASLt, bf16 output) on
    the decode projections of the Qwen3-8B and Qwen3-30B-A3B shapes, at batch
    heights 1..512, weights cold: each timed launch reads a different copy of
    the weight, with at least 1.2 GB of copies, so that no launch finds its
    weight in the L2 or the Infinity Cache.  Returns a markdown table."""
    import numpy as np
    import torch
    shapes = [("8B qkv", 6144, 4096), ("8B o", 4096, 4096), ("8B gate/up", 24576, 4096),
              ("8B down", 4096, 12288), ("8B lm head", 151936, 4096),
              ("30B-A3B qkv", 5120, 2048), ("30B-A3B o", 2048, 4096), ("30B-A3B lm head", 151936, 2048)]
    Ms = [1, 16, 64, 128, 256, 384, 512]
    lines = ["| projection (N x K) | rows | library us | hipBLASLt us | library / hipBLASLt time | "
             "library TFLOP/s | library weight GB/s |", "|---|---:|---:|---:|---:|---:|---:|"]
    tot_l = tot_t = 0.0
    for name, N, K in shapes:
        wb = N * K * 2
        ncopy = max(2, int(np.ceil(1.2e9 / wb)))
        W = []
        for i in range(ncopy):
            w = torch.empty(N * K, dtype=torch.bfloat16, device="cuda")
            B.darts_fill_uniform(w, 40 + i, 5, B.DARTS_BF16)
            W.append(w)
        A = torch.empty(512 * K, dtype=torch.bfloat16, device="cuda")
        B.darts_fill_uniform(A, 39, 5, B.DARTS_BF16)
        C = torch.empty(512 * N, dtype=torch.float32, device="cuda")
        for M in Ms:
            ws = torch.empty(max(B.darts_gemm_workspace_bytes(M, N, K), 256), dtype=torch.uint8, device="cuda")
            a2 = A[:M * K].view(M, K)
            it = max(ncopy, reps)

            def ours(j):
                B.darts_gemm(A, W[j % ncopy], C, M, N, K, B.DARTS_BF16, 0, ws)

            def theirs(j):
                torch.nn.functional.linear(a2, W[j % ncopy].view(N, K))

            res = []
            for fn in (ours, theirs):
                for j in range(ncopy):
                    fn(j)
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for j in range(it):
                    fn(j)
                e1.record()
                torch.cuda.synchronize()
                res.append(e0.elapsed_time(e1) * 1e3 / it)
            us, ref = res
            tot_l += us
            tot_t += ref
            lines.append(f"| {name} ({N} x {K}) | {M} | {us:.1f} | {ref:.1f} | {us / ref:.2f} | "
                         f"{2.0 * M * N * K / us / 1e6:.0f} | {wb / us / 1e3:.0f} |")
            print(f"[bench] gemm {name} M={M}: {us:.1f} us, hipBLASLt {ref:.1f} us", file=sys.stderr, flush=True)
        del W, A, C
        torch.cuda.empty_cache()
    lines.append(f"| all cases (sum of times) | | {tot_l:.0f} | {tot_t:.0f} | {tot_l / tot_t:.2f} | | |")
    return "\n".join(lines)


def launch_gap(B, n=1000, reps=3):
    """GPU time per kernel of a chain of n dependent one-block launches (the
    library's fill kernel over 1024 floats), launched one by one on a stream
    and replayed from a captured HIP graph.  Four 8 GiB streaming reads are
    queued first each time, so the host has queued the whole chain before the
    GPU reaches it and the figure is the device-side cost of a launch, not the
    host's launch rate.  Every graph replay's output is checked against the
    same fill done eagerly."""
    import torch
    s = torch.cuda.Stream()
    big = torch.zeros(8 << 30, dtype=torch.uint8, device="cuda")
    sink = torch.empty(8192, dtype=torch.float32, device="cuda")
    tiny = torch.zeros(1024, dtype=torch.float32, device="cuda")
    ref = torch.empty_like(tiny)
    out = {"chain": n}
    with torch.cuda.stream(s):
        B.darts_fill_uniform(ref, 7, 11, B.DARTS_F32)

        def fill_chain():
            for i in range(n):
                B.darts_fill_uniform(tiny, 7, 11, B.DARTS_F32)

        def timed(run):
            best = []
            for _ in range(reps):
                for _ in range(4):
                    B.darts_stream_read(big, sink)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(s)
                run()
                e1.record(s)
                s.synchronize()
                best.append(e0.elapsed_time(e1) * 1e3 / n)
            return min(best)

        out["stream_us_per_launch"] = timed(fill_chain)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            fill_chain()
        ok = True

        def replay():
            g.replay()

        out["graph_us_per_launch"] = timed(replay)
        for _ in range(3):
            tiny.zero_()
            g.replay()
            s.synchronize()
            ok = ok and bool(torch.equal(tiny, ref))
        out["graph_replays_match_eager"] = ok
    del big
    torch.cuda.empty_cache()
    return out


def kernel_sweep(B, steps, warmup):
    """Stateless kernels on the sweep's inputs (bf16, data seed 1): decode
    attention over 1024 trajectories with lognormal(1500, 1.0) contexts clipped
    to [16, 32768] in a shuffled page pool; the fused sampler on 1024 x 151936
    logits ~ N(0, 3); selection over 65536 trajectories in groups of 16."""
    import numpy as np
    import torch
    from workload import sweep_attention_inputs, sweep_sampler_logits, sweep_selection_inputs
    from workload.gen import sweep_page_table
    from workload.configs import SWEEP
    out = {"metric": "kernel sweep", "data": "synthetic (sweep inputs, seed 1)"}
    seed = SWEEP["seed"]
    hq, hkv, hd = SWEEP["attn_hq"], SWEEP["attn_hkv"], SWEEP["attn_hd"]
    ctx, rng = sweep_attention_inputs()
    pt, n_pages = sweep_page_table(ctx.astype(np.int64), 16, rng)
    rows = len(ctx)
    q = torch.empty(rows * hq * hd, dtype=torch.bfloat16, device="cuda")
    kp = torch.empty(n_pages * hkv * 16 * hd, dtype=torch.bfloat16, device="cuda")
    vp = torch.empty_like(kp)
    B.darts_fill_uniform(q, 0, seed, B.DARTS_BF16)
    B.darts_fill_kv_pool(kp, vp, n_pages, hkv, hd, seed, B.DARTS_BF16)
    ptd = torch.from_numpy(pt).cuda()
    ctxd = torch.from_numpy(ctx.astype(np.int32)).cuda()
    o = torch.empty_like(q)
    max_ctx = int(ctx.max())
    ws = torch.empty(B.darts_attn_workspace_bytes(rows, hq, hkv, hd, max_ctx), dtype=torch.uint8, device="cuda")
    alg = float(ctx.sum()) * hkv * hd * 2 * 2 + rows * 2 * hq * hd * 2 + float(np.ceil(ctx / 16).sum()) * 4

    def timed(fn, n):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(n):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n * 1e3   # us

    n = max(steps, 10)
    us = timed(lambda: B.darts_attn_decode(q, kp, vp, n_pages, ptd, ctxd, hq, hkv, hd, max_ctx,
                                           B.DARTS_BF16, o, ws), n)
    out["attention"] = {"rows": rows, "sum_ctx": int(ctx.sum()), "algorithmic_bytes": alg, "us": us,
                        "achieved_GBs": alg / (us * 1e-6) / 1e9,
                        "frac_of_hbm_peak": alg / (us * 1e-6) / 1e9 / HBM_PEAK_GBS}
    del kp, vp
    torch.cuda.empty_cache()
    rd = hbm_read_rate(B)
    out["hbm_read"] = {"GBs": rd, "frac_of_hbm_peak": rd / HBM_PEAK_GBS,
                       "kernel": "darts_stream_read over 8 GiB"}
    out["attention"]["frac_of_measured_read"] = out["attention"]["achieved_GBs"] / rd
    bits = sweep_sampler_logits()
    lg = torch.from_numpy(bits.view(np.int16)).cuda().view(torch.bfloat16)
    R, V = bits.shape
    traj = torch.arange(R, dtype=torch.int32, device="cuda")
    stp = torch.zeros(R, dtype=torch.int32, device="cuda")
    tok = torch.empty(R, dtype=torch.int32, device="cuda")
    lp = torch.empty(R, dtype=torch.float32, device="cuda")
    en = torch.empty(R, dtype=torch.float32, device="cuda")
    us = timed(lambda: B.darts_sample(lg, B.DARTS_BF16, seed, traj, stp, 1.0, None, tok, lp, en), n)
    out["sampler"] = {"rows": R, "vocab": V, "us": us, "logit_bytes": R * V * 2,
                      "achieved_GBs": R * V * 2 / (us * 1e-6) / 1e9}
    raw, mlp = sweep_selection_inputs()
    cap = SWEEP["sel_cap"]
    ln = np.minimum(raw, cap).astype(np.int32)
    st0 = np.where(raw > cap, 2, 1).astype(np.uint8)
    std = torch.from_numpy(st0).cuda()
    lnd = torch.from_numpy(ln).cuda()
    mld = torch.from_numpy(mlp).cuda()
    m, k = SWEEP["sel_m"], SWEEP["sel_k"]
    kept = torch.empty((len(ln) // m, k), dtype=torch.int32, device="cuda")
    comp = torch.empty(len(ln) // m, dtype=torch.uint8, device="cuda")
    us = timed(lambda: B.darts_select_groups(std, lnd, mld, m, k, 1, 2 * k, 1, kept, comp), n)
    out["selection"] = {"trajectories": len(ln), "groups": len(ln) // m, "us": us}
    # with page reclaim of the completed groups: the final step, every group
    # completes and frees all of its members' pages
    from workload.gen import sweep_selection_pages
    off, pages = sweep_selection_pages(ln)
    off_d, pages_d = torch.from_numpy(off).cuda(), torch.from_numpy(pages).cuda()
    free = torch.empty_like(pages_d)
    nfree = torch.zeros(1, dtype=torch.int32, device="cuda")
    work = torch.empty(len(ln) // m + 1, dtype=torch.int32, device="cuda")
    us = timed(lambda: B.darts_select_groups(std, lnd, mld, m, k, 1, 2 * k, 1, kept, comp, off_d, pages_d,
                                             free, nfree, work), n)
    torch.cuda.synchronize()
    out["selection_reclaim"] = {"trajectories": len(ln), "page_ids": len(pages),
                                "reclaimed": int(nfree.item()), "us": us,
                                "page_id_GBs": 2 * 4 * len(pages) / (us * 1e-6) / 1e9}
    return out


def next_rows(B, model, run, threshold):
    """The widened rows on one workload, each measured on the GPU:
    * adaptive redundancy (Alg. 1, App. B): a uniform rollout gives each
      prompt's length spread; the EMA of it (first observation as is)
      weights Alg. 1, which spreads the paper's solved budget of 1.5 N M
      candidates over M'_i in [M, 2M]; the planned rollout then runs on the
      same prompts and forced lengths;
    * token-chunk streaming: the uniform rollout again with chunks dispatched
      after every step once `threshold` tokens are pending (host copies of
      the descriptors and tokens included in the timed region);
    * group advantages (Eq. 2) of the uniform rollout's kept groups with
      Bernoulli(0.5) rewards.
    The allocation is measured on the configuration's own lengths (drawn
    alike for every prompt) and on lengths whose spread belongs to the prompt
    (alternating lognormal sigma 0.3 / 1.2, the tail only on the wide ones)."""
    import numpy as np
    import torch
    from workload import rollout_inputs
    prompts, forced = rollout_inputs(model, run)
    pr = torch.from_numpy(np.ascontiguousarray(prompts.reshape(-1))).cuda()
    fl = torch.from_numpy(forced.astype(np.int32)).cuda()
    P, m, k = run.n_prompts, run.m, run.k

    def progress(s, rows):
        if s % 1000 == 0:
            print(f"[bench]   step {s}: live {len(rows['traj'])}", file=sys.stderr, flush=True)

    def timed_rollout(lengths, flags=0, plan=None):
        ro = B.Rollout(model, run, flags=flags)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        st = ro.run_to_completion(pr, lengths, plan=plan, on_step=progress)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        print(f"[bench] next: rollout ({'planned' if plan is not None else 'uniform'}) {dt:.1f} s, "
              f"{st['steps']} steps", file=sys.stderr, flush=True)
        return ro, dt, st

    def allocation(lengths):
        """uniform M'_i = 2M, then the planned rollout on the same inputs"""
        ro, t_u, st_u = timed_rollout(lengths)
        lens = ro.traj_scores()[0].cpu().numpy()
        kept_u = ro.kept.clone()
        ro.close()
        # host planning, as an RL loop runs it between iterations
        t0 = time.perf_counter()
        sigma = B.darts_prompt_length_std(lens, None, P, m)
        est, seen = np.zeros(P), np.zeros(P, np.uint8)
        B.darts_ema_update(est, seen, sigma, 0.5)
        m_total = int(round(1.5 * P * k))
        plan = B.darts_allocate_redundancy(est, k, 2 * k, m_total, seen)
        plan_us = (time.perf_counter() - t0) * 1e6
        ro, t_p, st_p = timed_rollout(lengths, plan=plan)
        ro.close()
        return kept_u, t_u, {
            "uniform": {"candidates": P * m, "time_to_kept_set_s": t_u, "tokens": st_u["tokens_decoded"],
                        "steps": st_u["steps"]},
            "planned": {"budget": m_total, "candidates": int(plan.sum()),
                        "plan_histogram": {int(v): int((plan == v).sum()) for v in np.unique(plan)},
                        "planning_us": plan_us, "time_to_kept_set_s": t_p,
                        "tokens": st_p["tokens_decoded"], "steps": st_p["steps"],
                        "time_vs_uniform": t_p / t_u,
                        "tokens_vs_uniform": st_p["tokens_decoded"] / st_u["tokens_decoded"]}}

    out = {"metric": "widened rows: adaptive redundancy, token-chunk streaming, group advantages",
           "config": {"workload": workload_desc(model, run), "name": model.name}}
    kept, t_u, out["allocation_same_spread"] = allocation(fl)
    from workload.gen import heterogeneous_forced_lengths
    fh = torch.from_numpy(heterogeneous_forced_lengths(run, run.workload_seed + 100)).cuda()
    _, _, out["allocation_per_prompt_spread"] = allocation(fh)
    # streaming
    ro = B.Rollout(model, run, flags=B.FLAG_STREAM)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    n_disp = n_tok = 0
    ro.darts_prefill(pr, fl)
    ro.darts_select_and_prune()
    while True:
        done = ro.n_done >= P
        got = ro.stream_chunks(threshold, flush=done)
        if got is not None:
            n_disp += 1
            n_tok += len(got[1])
        if done:
            break
        ro.darts_decode_step()
        ro.darts_select_and_prune()
    torch.cuda.synchronize()
    t_s = time.perf_counter() - t0
    print(f"[bench] next: streaming rollout {t_s:.1f} s", file=sys.stderr, flush=True)
    st_s = ro.stats()
    ro.close()
    out["streaming"] = {"threshold_tokens": threshold, "dispatches": n_disp, "tokens_streamed": n_tok,
                        "tokens_decoded": st_s["tokens_decoded"], "time_to_kept_set_s": t_s,
                        "time_vs_uniform": t_s / t_u}
    # advantages of the kept groups
    rng = np.random.default_rng(0)
    reward = torch.from_numpy((rng.random(P * m) < 0.5).astype(np.float32)).cuda()
    adv = torch.empty((P, k), dtype=torch.float32, device="cuda")
    for _ in range(3):
        B.darts_group_advantages(kept, reward, adv)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(20):
        B.darts_group_advantages(kept, reward, adv)
    e1.record()
    torch.cuda.synchronize()
    out["advantages"] = {"groups": P, "k": k, "us": e0.elapsed_time(e1) / 20 * 1e3,
                         "finite": bool(torch.isfinite(adv).all().item())}
    return out


ATTN_SOURCES = ("paper_2605_30859_amd/csrc/k_attn.hip", "paper_2605_30859_amd/csrc/common.h")
EXPERT_SOURCES = ("paper_2605_30859_amd/csrc/k_gemm.hip", "paper_2605_30859_amd/csrc/k_moe.hip",
                  "paper_2605_30859_amd/csrc/common.h")


def source_hash(rels=ATTN_SOURCES):
    import hashlib
    h = hashlib.sha256()
    for rel in rels:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def attn_source_hash():
    return source_hash(ATTN_SOURCES)


def _counter_rows(d):
    """Per-dispatch counter sums from the one *_counter_collection.csv under d."""
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if len(files) != 1:
        raise SystemExit(f"expected one counter_collection.csv under {d}, found {len(files)}")
    per = {}
    with open(files[0]) as f:
        for r in csv.DictReader(f):
            key = int(r["Dispatch_Id"])
            name, v = r["Kernel_Name"], float(r["Counter_Value"])
            per[key] = (name, per.get(key, (name, 0.0))[1] + v)
    return list(per.values())


def _pmc_class(name):
    """Kernel class of a profiled dispatch: decode attention or one of the
    two grouped expert GEMMs, told apart by the epilogue template argument
    (3 = SwiGLU = gate/up, otherwise down): argument 7 of the LDS-tiled
    gemm_dma_grouped_kernel, argument 4 of gemm_wd_grouped_kernel."""
    import re
    if "attn_bf16" in name:
        return "attention"
    for kern, pos in (("gemm_dma_grouped_kernel", 6), ("gemm_wd_grouped_kernel", 3)):
        mt = re.search(kern + r"<([^>]*)>", name)
        if mt:
            args = [a.strip() for a in mt.group(1).split(",")]
            return "expert_gate_up" if len(args) > pos and args[pos] == "3" else "expert_down"
    return None


def summarize_pmc(d, name="attn"):
    """HBM traffic per launch of the decode-attention kernel (and, in MoE runs,
    of the grouped expert GEMMs) from rocprofv3 --pmc runs under d:
    pmc_copy_FETCH_SIZE / pmc_copy_WRITE_SIZE (bench.py --copy-calibration)
    and pmc_<name>_FETCH_SIZE / pmc_<name>_WRITE_SIZE (the rollout with a
    kernel-name filter), plus the rollout's bench line in d/bench_<name>.json.
    Each counter is scaled by what it reads for a plain 1 GiB device copy."""
    out = {"kernel": "attn_bf16_kernel + attn_bf16_db_kernel", "kernel_source_sha256": attn_source_hash()}
    cal = {}
    for c in ("FETCH_SIZE", "WRITE_SIZE"):
        rows = [v for n, v in _counter_rows(os.path.join(d, f"pmc_copy_{c}")) if "copyBuffer" in n]
        kib = sum(rows) / len(rows)
        cal[c] = {"KiB_per_1GiB_copy": kib, "scale": (1 << 30) / (kib * 1024.0), "copies": len(rows)}
    out["copy_calibration"] = cal
    with open(os.path.join(d, f"bench_{name}.json")) as f:
        line = [l for l in f.read().splitlines() if l.startswith("{")][-1]
    b = json.loads(line)
    out["workload"] = b["config"]["workload"]
    alg = {"attention": b["roofline"]["algorithmic_bytes_per_launch"]}
    for k, v in (b.get("roofline_moe_experts") or {}).items():
        alg[k] = v["algorithmic_bytes_per_launch"]
    per = {}
    for c, key in (("FETCH_SIZE", "fetch_bytes_per_launch"), ("WRITE_SIZE", "write_bytes_per_launch")):
        groups = {}
        for n, v in _counter_rows(os.path.join(d, f"pmc_{name}_{c}")):
            k = _pmc_class(n)
            if k:
                groups.setdefault(k, []).append(v)
        for k, vals in groups.items():
            e = per.setdefault(k, {})
            e[key] = sum(vals) / len(vals) * 1024.0 * cal[c]["scale"]
            e[f"launches_{c}"] = len(vals)
    for k, e in per.items():
        e["algorithmic_bytes_per_launch"] = alg.get(k)
        e["traffic_bytes_per_launch"] = e.get("fetch_bytes_per_launch", 0.0) + e.get("write_bytes_per_launch", 0.0)
        if alg.get(k):
            e["measured_over_algorithmic"] = e["traffic_bytes_per_launch"] / alg[k]
        if k != "attention":
            e["kernel_source_sha256"] = source_hash(EXPERT_SOURCES)
    out.update(per.get("attention", {}))
    out["kernels"] = per
    return out


def summarize_mfma(d):
    """MFMA utilisation of the GEMM kernels from one rocprofv3 --pmc pass
    under d collecting MfmaUtil (the busy cycles of the matrix cores over
    active cycles x SIMDs, per dispatch), MfmaFlopsBF16 and GRBM_GUI_ACTIVE,
    per kernel (template configuration) and over all of them, each dispatch
    weighted by its active cycles."""
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if len(files) != 1:
        raise SystemExit(f"expected one counter_collection.csv under {d}, found {len(files)}")
    per = {}
    with open(files[0]) as f:
        for r in csv.DictReader(f):
            key = int(r["Dispatch_Id"])
            e = per.setdefault(key, {"name": r["Kernel_Name"]})
            e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    by = {}
    for e in per.values():
        name = e["name"].split("(")[0].replace("void ", "").replace("darts::", "")
        k = by.setdefault(name, {"dispatches": 0, "gui": 0.0, "busy_weighted": 0.0, "bf16_flop": 0.0})
        g = e.get("GRBM_GUI_ACTIVE", 0.0)
        k["dispatches"] += 1
        k["gui"] += g
        k["busy_weighted"] += g * e.get("MfmaUtil", 0.0) / 100.0
        k["bf16_flop"] += e.get("MfmaFlopsBF16", 0.0)
    tot = {"dispatches": 0, "gui": 0.0, "busy_weighted": 0.0, "bf16_flop": 0.0}
    out = {"kernels": {}}
    for name, k in sorted(by.items(), key=lambda kv: -kv[1]["gui"]):
        for f in tot:
            tot[f] += k[f]
        out["kernels"][name] = {"dispatches": k["dispatches"], "active_cycles": k["gui"],
                                "mfma_util": k["busy_weighted"] / max(k["gui"], 1.0),
                                "bf16_flop": k["bf16_flop"]}
    out["all_gemm_kernels"] = {"dispatches": tot["dispatches"], "active_cycles": tot["gui"],
                               "mfma_util": tot["busy_weighted"] / max(tot["gui"], 1.0),
                               "bf16_flop": tot["bf16_flop"]}
    return out


def summarize_stats(path, top=16):
    """Markdown table of a rocprofv3 --stats kernel_stats.csv."""
    import csv
    with open(path) as f:
        rows = list(csv.DictReader(f))
    tot = sum(float(r["TotalDurationNs"]) for r in rows)
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    lines = ["| kernel | calls | total ms | avg us | share |", "|---|---:|---:|---:|---:|"]
    for r in rows[:top]:
        name = r["Name"].replace("|", "\\|")
        name = name if len(name) < 90 else name[:87] + "..."
        lines.append(f"| `{name}` | {int(r['Calls'])} | {float(r['TotalDurationNs']) / 1e6:.1f} | "
                     f"{float(r['AverageNs']) / 1e3:.1f} | {100 * float(r['TotalDurationNs']) / tot:.1f}% |")
    lines.append(f"| all kernels | {sum(int(r['Calls']) for r in rows)} | {tot / 1e6:.1f} | | 100% |")
    return "\n".join(lines)


def summarize_gaps(path):
    """GPU idle time of the last rollout in a rocprofv3 kernel_trace.csv: the
    window runs from its first prefill_pages_kernel to its last prune_kernel.
    Gaps from a prune_kernel up to the next step's first kernel (an embedding
    or page-allocation kernel) are step boundaries: the copies that follow
    the selection, the host's read of the live count and the queueing of the
    next step.  Every other gap lies between two kernels of one step."""
    import csv
    with open(path) as f:
        rows = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"])
                for r in csv.DictReader(f)]
    rows.sort()
    starts = [i for i, r in enumerate(rows) if "prefill_pages_kernel" in r[2]]
    if not starts:
        raise SystemExit("no prefill_pages_kernel in the trace")
    lo = starts[-1]
    hi = max(i for i, r in enumerate(rows) if "prune_kernel" in r[2] and i >= lo)
    win = rows[lo:hi + 1]
    busy = step_gap = intra_gap = 0
    n_steps = big = 0
    end = win[0][0]
    after_prune = False
    for s, e, name in win:
        if s > end:
            g = s - end
            if after_prune:
                step_gap += g
            else:
                intra_gap += g
            big += g > 50_000
        busy += max(0, e - max(s, end))
        end = max(end, e)
        if "prune_kernel" in name:
            after_prune = True
            n_steps += 1
        elif "embed" in name or "alloc_pages" in name:
            after_prune = False
    span = win[-1][1] - win[0][0]
    return {"kernels": len(win), "prune_launches": n_steps, "span_s": span / 1e9, "busy_s": busy / 1e9,
            "idle_s": (span - busy) / 1e9, "step_boundary_idle_s": step_gap / 1e9,
            "step_boundary_idle_us_per_step": step_gap / 1e3 / max(1, n_steps),
            "intra_step_idle_s": intra_gap / 1e9, "gaps_over_50us": big}


def measured_traffic(config, kernel="attention"):
    """Per-launch HBM bytes of a kernel from the committed counter summary, or
    None when there is none for this workload or the kernel's sources changed
    since the counters were taken."""
    p = os.path.join(ROOT, "profiles", f"attn_traffic_{config}_rollout.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        t = json.load(f)
    if kernel == "attention":
        if t.get("kernel_source_sha256") != attn_source_hash():
            return None
        return t["traffic_bytes_per_launch"]
    e = t.get("kernels", {}).get(kernel)
    if not e or e.get("kernel_source_sha256") != source_hash(EXPERT_SOURCES):
        return None
    return e["traffic_bytes_per_launch"]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="qwen3-30b-a3b",
                    help="workload (default: the Qwen3-30B-A3B-shaped MoE rollout, the largest that "
                         "fits one GPU)")
    ap.add_argument("--budget-s", type=float, default=420.0,
                    help="wall-time budget of the whole run: a step is one full rollout, so warmup is "
                         "clamped to 1 rollout and the timed rollouts to what fits (the line reports "
                         "the counts run next to the counts requested)")
    ap.add_argument("--timed-s", type=float, default=75.0,
                    help="target length of the timed region (at least one rollout is timed)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-abort", action="store_true", help="counterfactual without early stop")
    ap.add_argument("--cost-model-check", action="store_true",
                    help="after the timed rollouts, run the no-abort counterfactual once and compare its "
                         "measured decode time with Eq. 4 on the PTL curve fitted to the early-stop run")
    ap.add_argument("--next", action="store_true",
                    help="the widened rows instead of the benchmark: adaptive redundancy (Alg. 1) against "
                         "the uniform plan, token-chunk streaming, group advantages")
    ap.add_argument("--stream-threshold", type=int, default=16384)
    ap.add_argument("--shared-prefix", action="store_true",
                    help="decode attention reads each prompt's shared pages once per group")
    ap.add_argument("--sweep", action="store_true",
                    help="kernel sweep instead of the rollout: decode attention (1024 rows, 32/8 heads, "
                         "hd 128, lognormal contexts), fused sampler (1024 x 151936), selection (65536)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="three 1 GiB device copies (reference for HBM byte counters), then exit")
    ap.add_argument("--summarize-pmc", metavar="DIR",
                    help="print the traffic summary (JSON) of the rocprofv3 counter runs in DIR")
    ap.add_argument("--pmc-name", default="attn", help="run name of the counter directories in DIR")
    ap.add_argument("--summarize-mfma", metavar="DIR",
                    help="print the GEMM MFMA utilisation (JSON) of a rocprofv3 --pmc run in DIR")
    ap.add_argument("--summarize-stats", metavar="CSV",
                    help="print a markdown table of a rocprofv3 kernel_stats.csv")
    ap.add_argument("--step-log", metavar="JSONL",
                    help="write the last timed rollout's per-step metrics (live rows, device ms) "
                         "to this file, one JSON object a line")
    ap.add_argument("--launch-gap", action="store_true",
                    help="device-side cost per launch of a chain of dependent one-block kernels, "
                         "stream launches against a replayed HIP graph (JSON)")
    ap.add_argument("--gemm-compare", action="store_true",
                    help="time the library's GEMM against torch linear (hipBLASLt) on the decode "
                         "projections, weights cold; print a markdown table")
    ap.add_argument("--summarize-gaps", metavar="CSV",
                    help="print the GPU idle time (JSON) of the last rollout in a rocprofv3 kernel_trace.csv")
    args = ap.parse_args()
    if args.summarize_gaps:
        print(json.dumps(summarize_gaps(args.summarize_gaps), indent=1))
        return
    if args.summarize_pmc:
        print(json.dumps(summarize_pmc(args.summarize_pmc, args.pmc_name), indent=1))
        return
    if args.summarize_mfma:
        print(json.dumps(summarize_mfma(args.summarize_mfma), indent=1))
        return
    if args.summarize_stats:
        print(summarize_stats(args.summarize_stats))
        return
    if args.copy_calibration:
        import torch
        x = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
        y = torch.empty_like(x)
        x.fill_(1.0)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": 1 << 30, "copies": 3}))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the library runs the rollout of one data-parallel "
              "rank (prompt groups are independent); multi-GPU runs are not part of it.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2605_30859_amd import binding as B
    from workload import get_config, rollout_inputs

    torch.cuda.set_device(0)
    B.load_library()
    if args.sweep:
        print(json.dumps(kernel_sweep(B, args.steps, args.warmup)), flush=True)
        return
    if args.gemm_compare:
        print(gemm_compare(B), flush=True)
        return
    if args.launch_gap:
        print(json.dumps(launch_gap(B)), flush=True)
        return
    model, run = get_config(args.config)
    if args.next:
        print(json.dumps(next_rows(B, model, run, args.stream_threshold)), flush=True)
        return
    prompts, forced = rollout_inputs(model, run)
    flags = (B.FLAG_TIMING | B.FLAG_STEP_TIMES | (B.FLAG_NO_ABORT if args.no_abort else 0) |
             (B.FLAG_SHARED_PREFIX if args.shared_prefix else 0))
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

    # A step is a whole rollout (tens of seconds at the large configurations):
    # one warmup rollout at most, then as many timed rollouts as fit both the
    # timed-region target and what is left of the budget once the CPU
    # baseline and the read-rate probe are reserved.
    n_warm = min(max(args.warmup, 0), 1)
    t_roll = None
    for w in range(n_warm):
        dt, st = one_rollout()
        t_roll = dt
        print(f"[bench] warmup {w}: {dt:.2f} s, {st['tokens_decoded']} tokens", file=sys.stderr,
              flush=True)
    torch.cuda.synchronize()
    reserve = 0.0 if args.no_cpu_baseline else 45.0
    left = args.budget_s - (time.perf_counter() - T_PROCESS) - reserve - 15.0
    n_steps = max(1, args.steps)
    if t_roll is not None:
        n_steps = max(1, min(n_steps, int(min(args.timed_s, left) // t_roll)))
    print(f"[bench] timing {n_steps} rollout(s) ({args.steps} requested)", file=sys.stderr, flush=True)
    walls, stats = [], []
    t0 = time.perf_counter()
    for k in range(n_steps):
        dt, st = one_rollout()
        walls.append(dt)
        stats.append(st)
        print(f"[bench] step {k}: {dt:.2f} s, {st['tokens_decoded']} tokens, "
              f"{st['steps']} sampling steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    total = time.perf_counter() - t0
    n_timed = len(walls)
    tokens = sum(s["tokens_decoded"] for s in stats)
    attn_ms = sum(s["attn_ms"] for s in stats)
    attn_b = sum(s["attn_bytes"] for s in stats)
    attn_n = sum(s["attn_launches"] for s in stats)
    gemm_ms = sum(s["gemm_ms"] for s in stats)
    gemm_f = sum(s["gemm_flop"] for s in stats)
    ach = attn_b / (attn_ms * 1e-3) / 1e9 if attn_ms > 0 else 0.0
    peak_mm = BF16_PEAK_TFLOPS if model.dtype == "bf16" else FP32_PEAK_TFLOPS
    gemm_tf = gemm_f / (gemm_ms * 1e-3) / 1e12 if gemm_ms > 0 else 0.0
    # rollout cost model (Eq. 4) on this engine: PTL fitted to the last timed
    # rollout's per-step (live rows, device ms) samples
    rows, sms, pf_ms = ro.step_times()
    if args.step_log:
        # per-step metrics of the last timed rollout, one JSON object a line
        with open(args.step_log, "w") as f:
            f.write(json.dumps({"phase": "prefill", "device_ms": float(pf_ms)}) + "\n")
            for i, (nr, ms) in enumerate(zip(rows.tolist(), sms.tolist())):
                f.write(json.dumps({"phase": "decode", "step": i + 1, "live_rows": int(nr),
                                    "device_ms": float(ms)}) + "\n")
    lens = ro.traj_scores()[0].cpu().numpy()
    ptl = B.darts_fit_ptl(rows, sms.astype(np.float64))
    eq4 = B.darts_rollout_cost(np.maximum(lens[lens > 0] - 1, 0), ptl)
    cost_model = {"ptl_ms": {"b1": ptl[0], "b2": ptl[1], "c0": ptl[2], "c1": ptl[3], "c2": ptl[4],
                             "c3": ptl[5]},
                  "decode_steps": int(len(rows)), "decode_ms_measured": float(sms.sum()),
                  "decode_ms_eq4": eq4, "prefill_ms": pf_ms}
    cls = {}
    for i, name in enumerate(["qkv", "o", "gate_up", "down", "lm_head", "moe_block"]):
        ms = sum(s["gemm_cls_ms"][i] for s in stats)
        fl_ = sum(s["gemm_cls_flop"][i] for s in stats)
        cls[name] = {"ms": ms, "tflops": fl_ / (ms * 1e-3) / 1e12 if ms > 0 else 0.0}
    moe_roof = None
    if model.is_moe:
        # the grouped expert GEMMs inside the MoE block: algorithmic bytes (the
        # touched experts' weights once, routed rows in and out) over their own
        # HIP-event time
        moe_roof = {}
        for i, name in enumerate(["expert_gate_up", "expert_down"]):
            ms = sum(s["moe_expert_ms"][i] for s in stats)
            by = sum(s["moe_expert_bytes"][i] for s in stats)
            n_l = sum(s["moe_expert_launches"][i] for s in stats)
            ach_m = by / (ms * 1e-3) / 1e9 if ms > 0 else 0.0
            moe_roof[name] = {"bound": "hbm", "achieved": ach_m, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                              "frac": ach_m / HBM_PEAK_GBS, "traffic": measured_traffic(args.config, name),
                              "kernel": ("gemm_wd_grouped_kernel (gate/up + SwiGLU; gemm_dma_grouped_kernel "
                                         "below 2 and above 96 rows per expert)") if i == 0 else
                                        "gemm_dma_grouped_kernel (down)",
                              "launches": n_l, "avg_launch_us": 1e3 * ms / max(n_l, 1),
                              "algorithmic_bytes_per_launch": by / max(n_l, 1),
                              "share_of_step_time": ms * 1e-3 / total}
        cls["moe_block"]["routing_and_combine_ms"] = cls["moe_block"]["ms"] - sum(
            sum(s["moe_expert_ms"][i] for s in stats) for i in range(2))
    ro.close()
    try:
        read_gbs = hbm_read_rate(B)
    except Exception as e:  # reported next to the peak; never the metric itself
        print(f"[bench] read-rate probe failed: {e!r}", file=sys.stderr, flush=True)
        read_gbs = float("nan")
    roof = gemm_class_roofline(model, run, rows, HBM_PEAK_GBS, peak_mm)
    for name, rms in roof.items():
        if cls[name]["ms"] > 0:
            cls[name]["roofline_ms"] = rms
            cls[name]["frac_of_roofline"] = rms / cls[name]["ms"]
    bound_peak = rollout_bound(model, run, rows, HBM_PEAK_GBS, peak_mm)
    bound_read = rollout_bound(model, run, rows, read_gbs, peak_mm)
    if args.cost_model_check and not args.no_abort:
        ro2 = B.Rollout(model, run, flags=B.FLAG_STEP_TIMES | B.FLAG_NO_ABORT)
        ro2.run_to_completion(pr, fl)
        r2, ms2, _ = ro2.step_times()
        l2 = ro2.traj_scores()[0].cpu().numpy()
        ro2.close()
        cost_model["no_abort"] = {"decode_ms_measured": float(ms2.sum()),
                                  "decode_ms_eq4_from_early_stop_fit":
                                      B.darts_rollout_cost(np.maximum(l2[l2 > 0] - 1, 0), ptl),
                                  "decode_steps": int(len(r2))}

    out = {
        "metric": "rollout tokens/s + time-to-kept-set-complete; decode-attn HBM % of peak",
        "value": tokens / total,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": n_timed,
        "warmup": n_warm,
        "steps_requested": args.steps,
        "warmup_requested": args.warmup,
        "step_unit": "one whole rollout (prefill to the last kept set); warmup and timed rollouts are "
                     "clamped to the run's wall budget",
        "ms_per_step": 1e3 * total / n_timed,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": model.dtype,
        "data": "synthetic (seeded uniform prompt tokens, lognormal forced lengths, Philox random-init weights)",
        "config": {"workload": workload_desc(model, run), "name": args.config,
                   "prompts": run.n_prompts, "m": run.m, "k": run.k, "cap": run.cap,
                   "early_stop": not args.no_abort,
                   "decode_attention": "shared-prefix" if args.shared_prefix else "per-row"},
        "time_to_kept_set_s": float(np.mean(walls)),
        "tokens_per_rollout": stats[-1]["tokens_decoded"],
        "sampling_steps": stats[-1]["steps"],
        "pages_hwm": stats[-1]["pages_hwm"],
        "kv_pool_pages": stats[-1]["n_pages"],
        "roofline": {"bound": "hbm", "kernel": "attn_bf16_kernel + attn_bf16_db_kernel (paged GQA decode attention)",
                     "achieved": ach, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": ach / HBM_PEAK_GBS, "traffic": measured_traffic(args.config),
                     "launches": attn_n, "avg_launch_us": 1e3 * attn_ms / max(attn_n, 1),
                     "timed": "HIP events on the context stream around every launch of every 8th decode step",
                     "algorithmic_bytes_per_launch": attn_b / max(attn_n, 1),
                     "measured_read_GBs": read_gbs, "frac_of_measured_read": ach / read_gbs,
                     "share_of_step_time": attn_ms * 1e-3 / total},
        "roofline_moe_experts": moe_roof,
        "gemm": {"bound": "mfma", "achieved": gemm_tf, "peak": peak_mm, "unit": "TFLOP/s",
                 "frac": gemm_tf / peak_mm, "share_of_step_time": gemm_ms * 1e-3 / total,
                 "frac_of_roofline": (sum(v.get("roofline_ms", 0.0) for v in cls.values())
                                      / max(sum(v["ms"] for v in cls.values() if "roofline_ms" in v), 1e-9)),
                 "roofline_note": "per class: the schedule's max(FLOP / MFMA peak, weight bytes / HBM peak) "
                                  "summed over launches, over the measured class time",
                 "by_class": cls},
        "cost_model": cost_model,
        "rollout_bound": {
            "what": "roofline bound of the measured schedule (per step: KV bytes / HBM + max(weights / HBM, "
                    "GEMM FLOP / MFMA peak), plus the prefill)",
            "bound_s_at_peak": bound_peak, "tokens_per_s_at_peak": stats[-1]["tokens_decoded"] / bound_peak,
            "frac_at_peak": bound_peak / float(np.mean(walls)),
            "bound_s_at_measured_read": bound_read,
            "frac_at_measured_read": bound_read / float(np.mean(walls))},
        "cpu_baseline": None,
        "paper_context": "the paper reports end-to-end RL training speedups only: up to 1.77x over VeRL "
                         "(Sec. 5.2) on 8-node clusters of NVIDIA H20 GPUs, precision not stated; "
                         "context, not a figure for this metric",
    }
    if not args.no_cpu_baseline:
        try:
            out["cpu_baseline"] = cpu_baseline(model, run)
            try:
                gs = gpu_subset_rate(B, model, run)
                out["cpu_baseline"]["gpu_same_subset"] = gs
                out["cpu_baseline"]["gpu_over_oracle"] = gs["value"] / out["cpu_baseline"]["value"]
            except Exception as e:
                out["cpu_baseline"]["gpu_same_subset"] = {"error": repr(e)}
        except Exception as e:  # the baseline is context, never the product path
            out["cpu_baseline"] = {"error": repr(e)}
    out["wall_s"] = time.perf_counter() - T_PROCESS
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

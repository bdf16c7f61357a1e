"""MoE decoder on the GPU (route, grouped expert GEMMs, combine) against the
oracle: a reduced Qwen3-30B-A3B-like model, the full-width MoE layer end to
end (tokens and routing teacher-forced, every decoded row compared), and the
full-size configuration's schedule (steps, tokens, kept sets)."""
import sys
from dataclasses import replace

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import model as OM
from oracle.rollout import rollout, schedule_only
from workload import get_config, rollout_inputs
from workload.configs import ModelCfg

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def _run_gpu(model, run, prompts, forced, force_tokens=None, keep_logits=False, kv_fill=None):
    from paper_2605_30859_amd import binding as B
    B.load_library()
    ro = B.Rollout(model, run)
    if kv_fill is not None:
        ro.debug_fill_kv(kv_fill)
    pr = torch.from_numpy(np.ascontiguousarray(prompts.reshape(-1))).to(DEV)
    fl = torch.from_numpy(forced.astype(np.int32)).to(DEV)
    steps = []

    def force_fn(s):
        if force_tokens is None:
            return None
        f = np.full(run.n_prompts * run.m, -1, dtype=np.int32)
        for g, toks in force_tokens.items():
            if s < len(toks):
                f[g] = toks[s]
        return torch.from_numpy(f).to(DEV)

    def on_step(s, rows):
        rec = {k: v.cpu().numpy().copy() for k, v in rows.items()}
        if keep_logits:
            rec["logits"] = ro.debug_logits(max(len(rec["traj"]), run.n_prompts)).cpu().numpy().copy()
        steps.append(rec)

    stats = ro.run_to_completion(pr, fl, on_step=on_step, force_fn=force_fn)
    ln, slp, mlp, st = [t.cpu().numpy() for t in ro.traj_scores()]
    res = dict(steps=steps, stats=stats, kept=ro.kept.cpu().numpy(), done=ro.done_step.cpu().numpy(),
               length=ln, mean_lp=mlp)
    ro.close()
    return res


def small_moe():
    model = ModelCfg("moe-small", 2, 256, 4, 2, 64, 0, 512, "bf16", 21, rope_theta=1e6,
                     n_experts=16, top_k=4, expert_ffn=256)
    _, run = get_config("qwen3-30b-a3b")
    run = replace(run, n_prompts=2, prompt_len=32, m=8, k=4, cap=24, len_median=10.0, len_tail=False,
                  kv_pool_gb=0.0)
    return model, run


def test_moe_small_teacher_forced():
    """bf16 MoE: logits within 2e-2 of the row max on every step whose token's
    routing (every layer) is at least 1e-3 away from a top-k tie; routing
    decisions nearer a tie may legitimately differ between bf16 and float64."""
    model, run = small_moe()
    prompts, forced = rollout_inputs(model, run)
    say("moe-small: oracle")
    W = OM.init_weights(model)
    ref = rollout(model, W, prompts, forced, run.m, run.k, run.cap, run.sample_seed, keep_logits=True)
    say("moe-small: GPU")
    got = _run_gpu(model, run, prompts, forced, force_tokens=ref.tokens, keep_logits=True)
    checked = excused = 0
    worst = 0.0
    for s, rec in enumerate(got["steps"]):
        for r, g in enumerate(rec["traj"]):
            g = int(g)
            if ref.route_margins[g][s] < 1e-3:
                excused += 1
                continue
            row = r if s > 0 else g // run.m
            lg, lr = rec["logits"][row], ref.logits[g][s]
            dz = np.max(np.abs(lg - lr))
            scale = np.max(np.abs(lr))
            worst = max(worst, dz / scale)
            assert dz <= 2e-2 * scale, (s, g, dz / scale)
            checked += 1
    say(f"moe-small: {checked} rows checked, {excused} near-tie routing rows excused, worst {worst:.2e}")
    assert checked > 0.5 * (checked + excused)
    for i in range(run.n_prompts):
        assert got["done"][i] == ref.done_step[i]
    assert got["stats"]["steps"] == ref.steps and got["stats"]["pages_used"] == 0


@pytest.mark.parametrize("E,top_k,kv_fill", [(8, 1, None), (8, 8, None), (8, 1, 0xFF)])
def test_moe_routing_extremes_teacher_forced(E, top_k, kv_fill):
    """The two ends of the routing: top-1 (one expert per token, weight 1
    after renormalisation) and top-k = E (every expert takes every row, the
    weights are the whole softmax; 8 of the router's 128 padded rows are
    real).  bf16 MoE against the oracle under teacher forcing, as in the
    reduced test: logits within 2e-2 of the row max wherever the routing is
    at least 1e-3 from a top-k tie (with k = E there is no decision to tie,
    so every row is compared).  With kv_fill the KV pools start as NaN in
    every byte: the value slots of a freshly opened decode page past the
    context take part in the bf16 P.V product with weight 0, so the append
    that opens a page must clear them (a NaN there once reached the logits
    of every row on that page)."""
    model = ModelCfg(f"moe-e{E}-k{top_k}", 2, 256, 4, 2, 64, 0, 512, "bf16", 23, rope_theta=1e6,
                     n_experts=E, top_k=top_k, expert_ffn=256)
    _, run = get_config("qwen3-30b-a3b")
    run = replace(run, n_prompts=2, prompt_len=32, m=8, k=4, cap=20, len_median=10.0, len_tail=False,
                  kv_pool_gb=0.0)
    prompts, forced = rollout_inputs(model, run)
    say(f"moe E={E} top-{top_k}: oracle")
    W = OM.init_weights(model)
    ref = rollout(model, W, prompts, forced, run.m, run.k, run.cap, run.sample_seed, keep_logits=True)
    say(f"moe E={E} top-{top_k}: GPU")
    got = _run_gpu(model, run, prompts, forced, force_tokens=ref.tokens, keep_logits=True,
                   kv_fill=kv_fill)
    checked = excused = 0
    worst = 0.0
    for s, rec in enumerate(got["steps"]):
        for r, g in enumerate(rec["traj"]):
            g = int(g)
            row = r if s > 0 else g // run.m
            lg, lr = rec["logits"][row], ref.logits[g][s]
            assert np.all(np.isfinite(lg)), (s, g)
            if ref.route_margins[g][s] < 1e-3:
                excused += 1
                continue
            dz = np.max(np.abs(lg - lr))
            scale = np.max(np.abs(lr))
            worst = max(worst, dz / scale)
            assert dz <= 2e-2 * scale, (s, g, dz / scale)
            checked += 1
    say(f"moe E={E} top-{top_k}: {checked} rows checked, {excused} near-tie routing rows excused, "
        f"worst {worst:.2e}")
    if top_k == E:
        assert excused == 0
    assert checked > 0.5 * (checked + excused)
    for i in range(run.n_prompts):
        assert got["done"][i] == ref.done_step[i]
    assert got["stats"]["steps"] == ref.steps and got["stats"]["pages_used"] == 0


def test_moe_expert_kernel_paths_teacher_forced():
    """One rollout through every kernel path of the grouped expert GEMMs:
    16 experts top-4, 32 prompts x 8 trajectories, so the prefill has 256
    routed rows per expert (128-row tiled tiles), the first decode steps
    51-64 (96-row gate/up tiles, weights straight into registers), the
    middle 4-46 (64-row, weights into registers) and the last steps 1.25
    (64-row tiled tiles, strip-packed weights); down runs 128- and 64-row
    tiled tiles.  The whole batch decodes on the GPU; prompt 0 and prompt 23
    (the last to complete) are teacher-forced with the oracle's tokens and
    experts (oracle.forced, computed here), and every row of theirs is
    compared as in the full-width test: logits at 256 ids, row max and
    log-sum-exp within 2e-2 of max|z|, log-prob and entropy, the sampled
    token bit-exact on the GPU's own logits, the router's probabilities and
    own top-k."""
    from forced_parity import check_forced, run_forced
    from oracle.forced import reference_values
    from workload.gen import teacher_forcing_tokens
    model = ModelCfg("moe-paths", 2, 256, 4, 2, 64, 0, 512, "bf16", 29, rope_theta=1e6,
                     n_experts=16, top_k=4, expert_ffn=256)
    _, run = get_config("qwen3-30b-a3b")
    run = replace(run, n_prompts=32, prompt_len=32, m=8, k=4, cap=40, len_median=10.0, len_tail=False,
                  kv_pool_gb=0.0, workload_seed=8)
    prompts, forced = rollout_inputs(model, run)
    sched = schedule_only(forced, run.n_prompts, run.m, run.k, run.cap, run.prompt_len)
    length = np.asarray(sched["length"])
    E, k = model.n_experts, model.top_k
    per_expert = [int((length > s).sum()) * k / E for s in range(1, sched["steps"])]
    say(f"moe kernel paths: decode rows per expert {per_expert}")
    assert run.n_prompts * run.prompt_len * k / E > 96          # the prefill's 128-row tiles
    assert any(48 < x <= 96 for x in per_expert) and any(2 <= x <= 48 for x in per_expert)
    assert any(x < 2 for x in per_expert)
    last = int(np.argmax(sched["done_step"]))
    steps = int(sched["done_step"][last]) + 1
    say("moe kernel paths: oracle")
    tokens = teacher_forcing_tokens(model, run, steps)
    g = reference_values(model, run, prompts, forced, tokens, [0, last], steps)
    rec, strict, route = run_forced(model, run, prompts, forced, g, "moe kernel paths", strict_all=True)
    n = check_forced(model, run, g, rec, strict, route, "moe kernel paths")
    decoded = int(rec["seen"].sum())
    say(f"moe kernel paths: {n} of {decoded} decoded subset rows compared")
    assert decoded > 0 and n == decoded


def test_moe_full_size_schedule():
    """Qwen3-30B-A3B shape (48 layers, d 2048, 32/4 heads, 128 experts top-8,
    expert FFN 768, vocab 151936; 64 prompts x 512, m 16, k 8, cap 16384):
    the GPU rollout completes with the schedule the forced lengths imply and
    kept sets equal to the selection of its own scores."""
    model, run = get_config("qwen3-30b-a3b")
    prompts, forced = rollout_inputs(model, run)
    say("moe full size: GPU rollout")
    got = _run_gpu(model, run, prompts, forced)
    s = schedule_only(forced, run.n_prompts, run.m, run.k, run.cap, run.prompt_len,
                      mean_lp=got["mean_lp"])
    assert got["stats"]["steps"] == s["steps"]
    assert got["stats"]["tokens_decoded"] == s["tokens_decoded"]
    assert got["stats"]["pages_hwm"] == s["pages_hwm"]
    for i in range(run.n_prompts):
        assert list(got["kept"][i]) == s["kept"][i]
    ent = np.concatenate([r["entropy"] for r in got["steps"]])
    lp = np.concatenate([r["logprob"] for r in got["steps"]])
    assert np.isfinite(ent).all() and np.isfinite(lp).all()
    assert (ent >= 0).all() and (ent <= np.log(model.vocab) + 1e-3).all() and (lp <= 1e-5).all()


def test_moe_full_width_teacher_forced():
    """The MoE layer at the Qwen3-30B-A3B width (d 2048, 32/4 heads x 128,
    128 experts, top-8, expert FFN 768) with 2 layers and a 4096-token
    vocabulary: 2 prompts x 32 tokens, m = 16, k = 8, cap 20, the first 20
    generated tokens teacher-forced with a seeded token table and every row's
    routing forced to the oracle's experts, so every row the GPU decodes is
    compared (logits at 512 ids, row max, log-sum-exp, log-prob, entropy, the
    sampled token bit-exact on the GPU's own logits at every step), and the
    router's own top-8 equals the oracle's wherever the k / k+1 margin exceeds
    twice the measured router-probability deviation.  Early stop aborts
    members inside the window; the rows before it are all checked."""
    import os
    from forced_parity import check_forced, run_forced
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "forced_moe-full-width.npz")
    g = dict(np.load(path))
    model, run = get_config("moe-full-width")
    prompts, forced = rollout_inputs(model, run)
    rec, strict, route = run_forced(model, run, prompts, forced, g, "moe full width", strict_all=True)
    n = check_forced(model, run, g, rec, strict, route, "moe full width")
    decoded = int(rec["seen"].sum())
    say(f"moe full width: {n} of {decoded} decoded subset rows compared")
    assert decoded > 0 and n == decoded

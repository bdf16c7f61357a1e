"""Rollouts under an adaptive redundancy plan (Alg. 1 sizes M'_i in [k, m]) on
the GPU against the oracle: shortest-only groups (M'_i = m_up) and dual-end
groups (M'_i < m_up) decoded together in one ragged batch."""
import sys
from dataclasses import replace

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import model as OM
from oracle.allocation import allocate, length_std
from oracle.rollout import rollout, schedule_only
from oracle.selection import LIVE
from workload import get_config, rollout_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(*a):
    print(*a, flush=True)


def _b():
    from paper_2605_30859_amd import binding
    binding.load_library()
    return binding


def _plan_from_lengths(lengths, P, m, k, total):
    """Alg. 1 over the length spreads of a previous (uniform) rollout."""
    sig = [length_std(list(lengths[i * m:(i + 1) * m])) for i in range(P)]
    return allocate(sig, total, k, m)


def run_gpu(model, run, prompts, forced, plan, force_tokens=None):
    B = _b()
    ro = B.Rollout(model, run)
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
        steps.append({k: v.cpu().numpy().copy() for k, v in rows.items()})

    stats = ro.run_to_completion(pr, fl, on_step=on_step, force_fn=force_fn, plan=plan)
    ln, slp, mlp, st = [t.cpu().numpy() for t in ro.traj_scores()]
    res = dict(steps=steps, stats=stats, kept=ro.kept.cpu().numpy(), done=ro.done_step.cpu().numpy(),
               length=ln, mean_lp=mlp, status=st)
    ro.close()
    return res


def test_tiny_plan_parity():
    """fp32 tiny decoder, N = 4 prompts, m = 8, k = 4, budget 1.5 N k = 24:
    every step's rows, tokens, log-probs and entropies, and the final kept
    sets, completion steps, lengths, statuses and page counts match the
    oracle run with the same plan."""
    model, run = get_config("tiny")
    prompts, forced = rollout_inputs(model, run)
    W = OM.init_weights(model)
    P, m, k = run.n_prompts, run.m, run.k
    say("plan tiny: uniform oracle rollout for the length spreads")
    base = rollout(model, W, prompts, forced, m, k, run.cap, run.sample_seed)
    plan = _plan_from_lengths([base.length[g] for g in range(P * m)], P, m, k, total=int(1.5 * P * k))
    assert sum(plan) == 24 and min(plan) >= k and max(plan) <= m
    say(f"plan tiny: plan {plan}; oracle rollout under the plan")
    ref = rollout(model, W, prompts, forced, m, k, run.cap, run.sample_seed, alloc=plan)
    got = run_gpu(model, run, prompts, forced, plan, force_tokens=ref.tokens)
    exists = {i * m + j for i in range(P) for j in range(plan[i])}
    assert len(got["steps"][0]["traj"]) == sum(plan)
    for s, rec in enumerate(got["steps"]):
        for r, g in enumerate(rec["traj"]):
            g = int(g)
            assert g in exists
            assert rec["token"][r] == ref.tokens[g][s]
            assert abs(rec["logprob"][r] - ref.logprobs[g][s]) <= 1e-5
            assert abs(rec["entropy"][r] - ref.entropies[g][s]) <= 1e-5
            if ref.margins[g][s] >= 1e-4:
                assert rec["sampled"][r] == ref.sampled[g][s]
    assert got["stats"]["steps"] == ref.steps
    assert got["stats"]["tokens_decoded"] == ref.tokens_decoded
    assert got["stats"]["pages_hwm"] == ref.pages_hwm and got["stats"]["pages_used"] == 0
    for i in range(P):
        assert list(got["kept"][i]) == ref.kept[i]
        assert got["done"][i] == ref.done_step[i]
    for g in range(P * m):
        if g in exists:
            assert got["length"][g] == ref.length[g] and got["status"][g] == ref.status[g]
        else:
            assert got["length"][g] == 0 and got["status"][g] == 4


def test_dense_small_plan_schedule():
    """bf16 dense-small model (8 layers, d 1024, 32 prompts, m = 16, k = 8)
    under an Alg. 1 plan with budget 1.75 N k (12 groups reach m_up and run
    shortest-only, 20 run dual-end): steps, tokens, page high-water
    mark and kept sets equal the model-free schedule of the same plan (mean
    log-probs from the GPU break length ties)."""
    model, run = get_config("dense-small")
    run = replace(run, cap=1024)
    prompts, forced = rollout_inputs(model, run)
    P, m, k = run.n_prompts, run.m, run.k
    lengths = np.minimum(forced, run.cap)
    plan = _plan_from_lengths(lengths, P, m, k, total=int(1.75 * P * k))
    assert any(p == m for p in plan) and any(p < m for p in plan)
    say(f"plan dense-small: {sum(1 for p in plan if p == m)} shortest-only groups, "
        f"{sum(1 for p in plan if p < m)} dual-end groups")
    got = run_gpu(model, run, prompts, forced, plan)
    s = schedule_only(forced, P, m, k, run.cap, run.prompt_len, mean_lp=got["mean_lp"], alloc=plan)
    assert got["stats"]["steps"] == s["steps"]
    assert got["stats"]["tokens_decoded"] == s["tokens_decoded"]
    assert got["stats"]["pages_hwm"] == s["pages_hwm"] and got["stats"]["pages_used"] == 0
    for i in range(P):
        assert list(got["kept"][i]) == s["kept"][i]
    assert list(got["length"]) == s["length"]


def test_plan_errors_and_reset():
    B = _b()
    model, run = get_config("tiny")
    ro = B.Rollout(model, run)
    with pytest.raises(B.DartsError) as e:
        ro.darts_set_plan([run.k - 1] + [run.m] * (run.n_prompts - 1))
    assert e.value.status == B.DARTS_EINVAL
    with pytest.raises(B.DartsError) as e:
        ro.darts_set_plan([run.m + 1] * run.n_prompts)
    assert e.value.status == B.DARTS_EINVAL
    prompts, forced = rollout_inputs(model, run)
    pr = torch.from_numpy(np.ascontiguousarray(prompts.reshape(-1))).to(DEV)
    fl = torch.from_numpy(forced.astype(np.int32)).to(DEV)
    ro.darts_set_plan([run.k] * run.n_prompts)
    rows = ro.darts_prefill(pr, fl)
    assert len(rows["traj"]) == run.k * run.n_prompts
    with pytest.raises(B.DartsError) as e:
        ro.darts_set_plan([run.m] * run.n_prompts)
    assert e.value.status == B.DARTS_ESTATE
    ro.darts_reset()                       # restores the uniform plan
    rows = ro.darts_prefill(pr, fl)
    assert len(rows["traj"]) == run.m * run.n_prompts
    ro.close()


def test_step_times_and_cost_model_identity():
    """DARTS_FLAG_STEP_TIMES records one (rows, ms) sample per decode step whose
    row counts are the live counts the lengths imply; Eq. 4 with the PTL curve
    fitted to those samples reproduces their total (least squares with an
    intercept has zero-sum residuals), which checks the step accounting."""
    B = _b()
    model, run = get_config("dense-small")
    run = replace(run, cap=512)
    prompts, forced = rollout_inputs(model, run)
    ro = B.Rollout(model, run, flags=B.FLAG_STEP_TIMES)
    pr = torch.from_numpy(np.ascontiguousarray(prompts.reshape(-1))).to(DEV)
    fl = torch.from_numpy(forced.astype(np.int32)).to(DEV)
    st = ro.run_to_completion(pr, fl)
    rows, ms, pf = ro.step_times()
    ln = ro.traj_scores()[0].cpu().numpy()
    ro.close()
    assert len(rows) == st["steps"] - 1 and pf > 0 and (ms > 0).all()
    exp_rows = [int((ln >= s).sum()) for s in range(2, st["steps"] + 1)]
    assert list(rows) == exp_rows
    p = B.darts_fit_ptl(rows, ms.astype(np.float64))
    T = B.darts_rollout_cost(np.maximum(ln - 1, 0), p)
    say(f"step times: {len(rows)} decode steps, {ms.sum():.1f} ms measured, Eq. 4 {T:.1f} ms; "
        f"prefill {pf:.2f} ms; PTL {p}")
    assert T == pytest.approx(float(ms.astype(np.float64).sum()), rel=1e-6)

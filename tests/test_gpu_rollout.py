"""End-to-end rollout parity on the GPU through the C ABI.

The oracle runs the rollout free (its own float64 logits, float32 Gumbel-max
decisions); the GPU is teacher-forced with the oracle's token history, so both
sides see the same prefixes.  Compared per step: the GPU's own sampled token
(bit-exact wherever the oracle's top-2 perturbed-score margin is at least tau),
logits, log-prob and entropy (tolerances in each test), the finished flags;
at the end: kept sets, completion steps, lengths, page counts."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import model as OM
from oracle.rollout import rollout, schedule_only
from oracle.sampler import sample_row
from oracle.selection import LIVE, EOS, TRUNC, ABORTED
from workload import get_config, rollout_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _b():
    from paper_2605_30859_amd import binding
    binding.load_library()
    return binding


def run_gpu(model, run, prompts, forced, force_tokens=None, flags=0, perm_seed=0, keep_logits=False,
            kv_pool_bytes=None, kv_fill=None):
    B = _b()
    ro = B.Rollout(model, run, flags=flags, page_perm_seed=perm_seed, kv_pool_bytes=kv_pool_bytes)
    if kv_fill is not None:
        ro.debug_fill_kv(kv_fill)
    pr = torch.from_numpy(np.ascontiguousarray(prompts.reshape(-1))).to(DEV)
    fl = torch.from_numpy(forced.astype(np.int32)).to(DEV)
    steps = []
    hwm_trace = []

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
            n = len(rec["traj"])
            rec["logits"] = ro.debug_logits(max(n, run.n_prompts)).cpu().numpy().copy()
        steps.append(rec)

    stats = ro.run_to_completion(pr, fl, on_step=on_step, force_fn=force_fn)
    ln, slp, mlp, st = [t.cpu().numpy() for t in ro.traj_scores()]
    res = dict(steps=steps, stats=stats, kept=ro.kept.cpu().numpy(), done=ro.done_step.cpu().numpy(),
               length=ln, sum_lp=slp, mean_lp=mlp, status=st)
    ro.close()
    return res


@pytest.fixture(scope="module")
def tiny():
    model, run = get_config("tiny")
    prompts, forced = rollout_inputs(model, run)
    say("tiny: oracle rollout")
    W = OM.init_weights(model)
    ref = rollout(model, W, prompts, forced, run.m, run.k, run.cap, run.sample_seed, keep_logits=True)
    say("tiny: GPU rollout (teacher-forced)")
    got = run_gpu(model, run, prompts, forced, force_tokens=ref.tokens, keep_logits=True)
    return model, run, prompts, forced, ref, got


def test_tiny_schedule_and_kept_sets(tiny):
    model, run, prompts, forced, ref, got = tiny
    assert got["stats"]["steps"] == ref.steps
    assert got["stats"]["tokens_decoded"] == ref.tokens_decoded
    assert got["stats"]["pages_hwm"] == ref.pages_hwm
    assert got["stats"]["pages_used"] == 0
    for i in range(run.n_prompts):
        assert list(got["kept"][i]) == ref.kept[i]
        assert got["done"][i] == ref.done_step[i]
    for g in range(run.n_prompts * run.m):
        assert got["length"][g] == ref.length[g]
        assert got["status"][g] == ref.status[g]


def test_tiny_per_step_parity(tiny):
    """fp32 configuration: logits within 1e-5 (relative to the row's max |logit|),
    log-prob and entropy within 1e-5 absolute, sampled tokens bit-exact where
    the oracle's top-2 Gumbel margin is >= 1e-4."""
    model, run, prompts, forced, ref, got = tiny
    excused = mism = checked = 0
    for s, rec in enumerate(got["steps"]):
        for r, g in enumerate(rec["traj"]):
            g = int(g)
            assert s < len(ref.tokens[g])
            lg_ref = ref.logits[g][s]
            row = r if s > 0 else g // run.m
            lg = rec["logits"][row]
            scale = max(1.0, np.max(np.abs(lg_ref)))
            assert np.max(np.abs(lg - lg_ref)) <= 1e-5 * scale, (s, g)
            assert abs(rec["logprob"][r] - ref.logprobs[g][s]) <= 1e-5, (s, g)
            assert abs(rec["entropy"][r] - ref.entropies[g][s]) <= 1e-5, (s, g)
            assert rec["token"][r] == ref.tokens[g][s]
            checked += 1
            if rec["sampled"][r] != ref.sampled[g][s]:
                if ref.margins[g][s] < 1e-4:
                    excused += 1
                else:
                    mism += 1
            fin = rec["finished"][r]
            exp_fin = 0
            if s == len(ref.tokens[g]) - 1 and ref.status[g] in (EOS, TRUNC):
                exp_fin = 1 if ref.status[g] == EOS else 2
            assert fin == exp_fin, (s, g, fin, exp_fin)
    say(f"tiny: {checked} rows checked, {excused} near-tie tokens excused")
    assert mism == 0
    assert excused <= max(1, checked // 1000)


def test_tiny_scores(tiny):
    model, run, prompts, forced, ref, got = tiny
    for g in range(run.n_prompts * run.m):
        assert abs(got["sum_lp"][g] - ref.sum_lp32[g]) <= 1e-4
        assert abs(got["mean_lp"][g] - ref.mean_lp32[g]) <= 1e-5


def test_tiny_free_running_matches_forced(tiny):
    """Without teacher forcing the GPU follows its own samples; with fp32
    parity this reproduces the oracle's token history exactly."""
    model, run, prompts, forced, ref, got = tiny
    free = run_gpu(model, run, prompts, forced)
    for s, rec in enumerate(free["steps"]):
        for r, g in enumerate(rec["traj"]):
            assert rec["token"][r] == ref.tokens[int(g)][s]


def test_determinism_and_page_permutation(tiny):
    """Two runs are bitwise identical, and a permuted initial free list (other
    physical page ids) changes no output."""
    model, run, prompts, forced, ref, got = tiny
    a = run_gpu(model, run, prompts, forced)
    b = run_gpu(model, run, prompts, forced, flags=_b().FLAG_PERMUTE_PAGES, perm_seed=12345)
    for x, y in zip(a["steps"], b["steps"]):
        for key in ("traj", "token", "sampled", "finished"):
            assert np.array_equal(x[key], y[key])
        for key in ("logprob", "entropy"):
            assert np.array_equal(x[key].view(np.uint32), y[key].view(np.uint32))
    assert np.array_equal(a["kept"], b["kept"])


def _same_steps(a, b, keys=("traj", "token", "sampled", "finished")):
    assert len(a["steps"]) == len(b["steps"])
    for s, (x, y) in enumerate(zip(a["steps"], b["steps"])):
        for key in keys:
            assert np.array_equal(x[key], y[key]), (s, key)
        for key in ("logprob", "entropy"):
            assert np.array_equal(x[key].view(np.uint32), y[key].view(np.uint32)), (s, key)
        if "logits" in x:
            assert np.array_equal(x["logits"].view(np.uint32), y["logits"].view(np.uint32)), s
    assert np.array_equal(a["kept"], b["kept"])


def test_tiny_pool_contents_do_not_matter(tiny):
    """KV pools holding NaN in every byte before the prefill (as memory left
    by earlier work may) change no output: every value the decode reads is
    one the rollout wrote."""
    model, run, prompts, forced, ref, got = tiny
    p = run_gpu(model, run, prompts, forced, force_tokens=ref.tokens, keep_logits=True, kv_fill=0xFF)
    _same_steps(got, p)


def test_no_abort_counterfactual(tiny):
    model, run, prompts, forced, ref, got = tiny
    B = _b()
    na = run_gpu(model, run, prompts, forced, flags=B.FLAG_NO_ABORT)
    mlp = np.array([ref.mean_lp32[g] for g in range(run.n_prompts * run.m)], np.float32)
    s = schedule_only(forced, run.n_prompts, run.m, run.k, run.cap, run.prompt_len, mean_lp=mlp,
                      early_stop=False)
    assert na["stats"]["steps"] == s["steps"]
    assert na["stats"]["tokens_decoded"] == s["tokens_decoded"]
    assert na["stats"]["pages_hwm"] == s["pages_hwm"]
    for i in range(run.n_prompts):
        assert list(na["kept"][i]) == s["kept"][i]


def test_dual_mode_tiny():
    """m < m_up: every group runs dual-end selection (K shortest + L longest valid)."""
    from dataclasses import replace
    model, run = get_config("tiny")
    run = replace(run, m_up=9, cap=40)
    prompts, forced = rollout_inputs(model, run)
    got = run_gpu(model, run, prompts, forced)
    s = schedule_only(forced, run.n_prompts, run.m, run.k, run.cap, run.prompt_len,
                      mean_lp=got["mean_lp"], m_up=9)
    assert got["stats"]["steps"] == s["steps"]
    assert got["stats"]["tokens_decoded"] == s["tokens_decoded"]
    for i in range(run.n_prompts):
        assert list(got["kept"][i]) == s["kept"][i]
    assert got["stats"]["pages_used"] == 0


@pytest.mark.parametrize("shape", [
    # (layers, d, hq, hkv, hd, ffn, vocab, prompts, prompt_len, m, k, cap, m_up)
    (3, 64, 4, 1, 128, 256, 1000, 3, 32, 6, 3, 40, None),      # GQA 4:1, hd 128, hq*hd != d
    (2, 96, 8, 2, 64, 192, 768, 2, 16, 5, 3, 48, None),        # m < 2k: dual-end groups
    (1, 128, 2, 2, 32, 512, 516, 5, 48, 4, 4, 30, None),       # k = m (no redundancy), 3 prompt pages
    (2, 128, 16, 4, 32, 256, 4096, 2, 16, 8, 2, 64, 9),        # G = 4 with 16 q heads, dual-end forced (m_up 9 > m)
])
def test_fp32_shape_variants(shape):
    """fp32 models of other shapes than the tiny configuration through the
    whole rollout (teacher-forced): schedule, kept sets, lengths and statuses
    equal the oracle's; per step log-probs and entropies within 1e-5, tokens
    bit-exact where the oracle's top-2 margin is at least 1e-4."""
    from workload.configs import ModelCfg, RunCfg
    L_, d, hq, hkv, hd, F, V, P, Lp, m, k, cap, m_up = shape
    model = ModelCfg("fp32-variant", L_, d, hq, hkv, hd, F, V, "f32", 11)
    run = RunCfg(P, Lp, m, k, cap, 16.0, 0.9, False, 5, 5, m_up=m_up)
    say(f"fp32 variant {shape}: oracle")
    prompts, forced = rollout_inputs(model, run)
    W = OM.init_weights(model)
    ref = rollout(model, W, prompts, forced, run.m, run.k, run.cap, run.sample_seed, m_up=run.m_up_eff)
    say(f"fp32 variant {shape}: GPU")
    got = run_gpu(model, run, prompts, forced, force_tokens=ref.tokens)
    assert got["stats"]["steps"] == ref.steps
    assert got["stats"]["tokens_decoded"] == ref.tokens_decoded
    assert got["stats"]["pages_hwm"] == ref.pages_hwm and got["stats"]["pages_used"] == 0
    for i in range(run.n_prompts):
        assert list(got["kept"][i]) == ref.kept[i], i
        assert got["done"][i] == ref.done_step[i], i
    for g in range(run.n_prompts * run.m):
        assert got["length"][g] == ref.length[g] and got["status"][g] == ref.status[g], g
    mism = 0
    for st, rec in enumerate(got["steps"]):
        for r, g in enumerate(rec["traj"]):
            g = int(g)
            assert abs(rec["logprob"][r] - ref.logprobs[g][st]) <= 1e-5, (st, g)
            assert abs(rec["entropy"][r] - ref.entropies[g][st]) <= 1e-5, (st, g)
            if rec["sampled"][r] != ref.sampled[g][st] and ref.margins[g][st] >= 1e-4:
                mism += 1
    assert mism == 0


def test_error_paths():
    B = _b()
    model, run = get_config("tiny")
    ro = B.Rollout(model, run)
    with pytest.raises(B.DartsError) as e:
        ro.darts_decode_step()
    assert e.value.status == B.DARTS_ESTATE
    with pytest.raises(B.DartsError) as e:
        ro.darts_select_and_prune()
    assert e.value.status == B.DARTS_ESTATE
    ro.close()
    # a pool too small for the first decode step's pages
    prompts, forced = rollout_inputs(model, run)
    page_bytes = model.n_layers * model.n_kv_heads * 16 * model.head_dim * 2 * 4
    ro = B.Rollout(model, run, kv_pool_bytes=page_bytes * (run.n_prompts + 5))
    pr = torch.from_numpy(prompts.reshape(-1).copy()).to(DEV)
    fl = torch.from_numpy(forced.astype(np.int32)).to(DEV)
    ro.darts_prefill(pr, fl)
    ro.darts_select_and_prune()
    with pytest.raises(B.DartsError) as e:
        ro.darts_decode_step()
    assert e.value.status == B.DARTS_ENOMEM
    st = ro.stats()
    assert st["steps"] == 1 and st["pages_used"] == run.n_prompts
    ro.close()


@pytest.fixture(scope="module")
def dense_small_reduced():
    """dense-small's model (8 layers, d 1024, 16/4 heads, hd 64, FFN 4096,
    V 32000, bf16) on 2 prompts of 32 tokens, m=16, k=8, cap 48."""
    from dataclasses import replace
    model, run = get_config("dense-small")
    run = replace(run, n_prompts=2, prompt_len=32, cap=48, len_median=20.0, kv_pool_gb=0.0)
    prompts, forced = rollout_inputs(model, run)
    say("dense-small reduced: oracle")
    W = OM.init_weights(model)
    ref = rollout(model, W, prompts, forced, run.m, run.k, run.cap, run.sample_seed, keep_logits=True)
    say("dense-small reduced: GPU")
    got = run_gpu(model, run, prompts, forced, force_tokens=ref.tokens, keep_logits=True)
    return model, run, ref, got


def _check_bf16(name, run, ref, got):
    """bf16 configuration: logits within 2e-2 of the row's max |logit|; the
    log-prob / entropy deviation is bounded by the logit deviation (|d lp| <= 2 max|d z|);
    sampled tokens bit-exact where the top-2 margin is >= 0.1."""
    excused = mism = checked = 0
    worst = 0.0
    for s, rec in enumerate(got["steps"]):
        for r, g in enumerate(rec["traj"]):
            g = int(g)
            row = r if s > 0 else g // run.m
            lg = rec["logits"][row]
            lg_ref = ref.logits[g][s]
            dz = np.max(np.abs(lg - lg_ref))
            scale = np.max(np.abs(lg_ref))
            worst = max(worst, dz / scale)
            assert dz <= 2e-2 * scale, (s, g, dz, scale)
            assert abs(rec["logprob"][r] - ref.logprobs[g][s]) <= 2 * dz + 1e-3
            assert abs(rec["entropy"][r] - ref.entropies[g][s]) <= 2 * dz + 1e-3
            checked += 1
            if rec["sampled"][r] != ref.sampled[g][s]:
                if ref.margins[g][s] < 0.1:
                    excused += 1
                else:
                    mism += 1
    say(f"{name}: {checked} rows, worst logit dev {worst:.3e}, {excused} excused")
    assert mism == 0
    assert excused <= checked // 5
    # given the same logits (the GPU's own), the sample is the oracle
    # sampler's and the log-prob and entropy are its values within 1e-3
    dlp_own = dent_own = 0.0
    n_own = 0
    for s, rec in enumerate(got["steps"]):
        for r in range(min(4, len(rec["traj"]))):
            g = int(rec["traj"][r])
            row = r if s > 0 else g // run.m
            tok, lp_o, ent_o = sample_row(rec["logits"][row], run.temperature, g, s, run.sample_seed,
                                          force=int(rec["token"][r]))
            assert tok == rec["sampled"][r], (s, g)
            dlp_own = max(dlp_own, abs(float(rec["logprob"][r]) - lp_o))
            dent_own = max(dent_own, abs(float(rec["entropy"][r]) - ent_o))
            n_own += 1
    say(f"{name}: on the GPU's own logits ({n_own} rows): |d logprob| worst {dlp_own:.3e}, "
        f"|d entropy| worst {dent_own:.3e}")
    assert dlp_own <= 1e-3 and dent_own <= 1e-3
    for i in range(run.n_prompts):
        assert got["done"][i] == ref.done_step[i]
    assert got["stats"]["steps"] == ref.steps
    assert got["stats"]["pages_used"] == 0


def test_dense_small_bf16_parity(dense_small_reduced):
    model, run, ref, got = dense_small_reduced
    _check_bf16("dense-small", run, ref, got)


def test_dense_small_bf16_pool_contents_do_not_matter(dense_small_reduced):
    """bf16: the value slots of a decode page past the context enter the
    P.V product with weight 0; with the pools NaN in every byte before the
    prefill, the append that opens a page clears them, and every output is
    bit for bit that of the run on fresh pools."""
    model, run, ref, got = dense_small_reduced
    prompts, forced = rollout_inputs(model, run)
    p = run_gpu(model, run, prompts, forced, force_tokens=ref.tokens, keep_logits=True, kv_fill=0xFF)
    _same_steps(got, p)


@pytest.fixture(scope="module")
def dense_small_prompt256():
    """dense-small's model on 2 prompts of 256 tokens (16 shared prompt pages
    each), m=16, k=8, cap 48; the GPU runs twice: with the shared-prefix decode
    attention and with the per-row kernel (which splits each row's 17-19 pages
    into chunks that the combine kernel merges: 32 rows x 4 kv heads leave
    most of the GPU idle otherwise)."""
    from dataclasses import replace
    model, run = get_config("dense-small")
    run = replace(run, n_prompts=2, prompt_len=256, cap=48, len_median=20.0, kv_pool_gb=0.0)
    prompts, forced = rollout_inputs(model, run)
    say("dense-small prompt 256: oracle")
    W = OM.init_weights(model)
    ref = rollout(model, W, prompts, forced, run.m, run.k, run.cap, run.sample_seed, keep_logits=True)
    B = _b()
    say("dense-small prompt 256: GPU, shared prefix")
    shared = run_gpu(model, run, prompts, forced, force_tokens=ref.tokens, keep_logits=True,
                     flags=B.FLAG_SHARED_PREFIX)
    say("dense-small prompt 256: GPU, per-row attention")
    rows = run_gpu(model, run, prompts, forced, force_tokens=ref.tokens, keep_logits=True)
    return run, ref, shared, rows


def test_dense_small_shared_prefix_parity(dense_small_prompt256):
    run, ref, shared, rows = dense_small_prompt256
    _check_bf16("dense-small prompt 256, shared prefix", run, ref, shared)


def test_dense_small_chunked_rows_parity(dense_small_prompt256):
    run, ref, shared, rows = dense_small_prompt256
    _check_bf16("dense-small prompt 256, per-row attention", run, ref, rows)


def test_qwen3_8b_full_size_schedule():
    """Qwen3-8B shape at full size (36 layers, d 4096, 32/8 heads x 128, FFN
    12288, vocab 151936; 32 prompts x 512, m 16, k 8, cap 8192), in the launch
    configuration the benchmark times: the rollout completes with the steps,
    tokens and page high-water mark the forced lengths imply, kept sets equal
    the selection of its own scores, every score is a valid log-prob /
    entropy, and a second run on a permuted page pool is bitwise identical."""
    model, run = get_config("qwen3-8b")
    prompts, forced = rollout_inputs(model, run)
    say("qwen3-8b full size: GPU rollout")
    got = run_gpu(model, run, prompts, forced)
    s = schedule_only(forced, run.n_prompts, run.m, run.k, run.cap, run.prompt_len,
                      mean_lp=got["mean_lp"])
    assert got["stats"]["steps"] == s["steps"]
    assert got["stats"]["tokens_decoded"] == s["tokens_decoded"]
    assert got["stats"]["pages_hwm"] == s["pages_hwm"] and got["stats"]["pages_used"] == 0
    for i in range(run.n_prompts):
        assert list(got["kept"][i]) == s["kept"][i]
    assert list(got["length"]) == s["length"]
    ent = np.concatenate([r["entropy"] for r in got["steps"]])
    lp = np.concatenate([r["logprob"] for r in got["steps"]])
    assert np.isfinite(ent).all() and np.isfinite(lp).all()
    assert (ent >= 0).all() and (ent <= np.log(model.vocab) + 1e-3).all() and (lp <= 1e-5).all()
    # reproducible at full size, whatever the physical pages: a second run
    # with a permuted free list gives bitwise the same scores and kept sets
    say("qwen3-8b full size: second GPU rollout, permuted page pool")
    again = run_gpu(model, run, prompts, forced, perm_seed=7)
    for key in ("length", "sum_lp", "mean_lp", "status", "kept", "done"):
        assert np.array_equal(np.asarray(again[key]).view(np.uint8), np.asarray(got[key]).view(np.uint8)), key
    assert again["stats"]["steps"] == got["stats"]["steps"]


def test_dense_small_full_config_prompt_prefix():
    """dense-small at its full configuration (32 prompts x 256 tokens, m=16,
    k=8, cap 4096, 512 rows per step), in the launch configuration the
    benchmark would use: the GPU decodes the whole batch while the oracle
    follows one prompt's group (its trajectories teacher-forced) for the
    prefill and the first 47 decode steps.  On that group: logits within 2e-2
    of the row's max on sampled steps, log-prob / entropy within twice the
    logit deviation there and within 0.25 everywhere, sampled tokens
    bit-exact where the top-2 margin is >= 0.1."""
    model, run = get_config("dense-small")
    prompts, forced = rollout_inputs(model, run)
    P, m, S = run.n_prompts, run.m, 48
    p = 18                                   # the group that completes first
    say("dense-small full config: oracle, prompt 18, 48 steps")
    W = OM.init_weights(model)
    ref = rollout(model, W, prompts, forced, m, run.k, run.cap, run.sample_seed, prompt_ids=[p],
                  keep_logits=True, max_steps=S)
    B = _b()
    ro = B.Rollout(model, run)
    pr = torch.from_numpy(np.ascontiguousarray(prompts.reshape(-1))).to(DEV)
    fl = torch.from_numpy(forced.astype(np.int32)).to(DEV)
    grp = list(range(p * m, (p + 1) * m))

    def force(s):
        f = np.full(P * m, -1, dtype=np.int32)
        for g in grp:
            if s < len(ref.tokens[g]):
                f[g] = ref.tokens[g][s]
        return torch.from_numpy(f).to(DEV)

    logit_steps = {0, 1, 16, S - 1}
    say("dense-small full config: GPU")
    recs = []
    rows = ro.darts_prefill(pr, fl, force(0))
    for s in range(S):
        if s > 0:
            rows = ro.darts_decode_step(force(s))
        rec = {k: v.cpu().numpy().copy() for k, v in rows.items()}
        if s in logit_steps:
            n = len(rec["traj"])
            lg = ro.debug_logits(max(n, P))
            sel = [p] if s == 0 else [r for r, g in enumerate(rec["traj"]) if g // m == p]
            rec["logits"] = {r: lg[r].cpu().numpy().copy() for r in sel}
        recs.append(rec)
        ro.darts_select_and_prune()
    assert ro.n_live > 0
    ro.close()
    checked = excused = 0
    for s, rec in enumerate(recs):
        for r, g in enumerate(rec["traj"]):
            g = int(g)
            if g // m != p or s >= len(ref.logprobs[g]):
                continue
            assert abs(rec["logprob"][r] - ref.logprobs[g][s]) <= 0.25
            assert abs(rec["entropy"][r] - ref.entropies[g][s]) <= 0.25
            if s in logit_steps:
                lg = rec["logits"][p if s == 0 else r]
                lr = ref.logits[g][s]
                dz = np.max(np.abs(lg - lr))
                assert dz <= 2e-2 * np.max(np.abs(lr)), (s, g)
                assert abs(rec["logprob"][r] - ref.logprobs[g][s]) <= 2 * dz + 1e-3
                assert abs(rec["entropy"][r] - ref.entropies[g][s]) <= 2 * dz + 1e-3
            if rec["sampled"][r] != ref.sampled[g][s]:
                assert ref.margins[g][s] < 0.1, (s, g)
                excused += 1
            checked += 1
    say(f"dense-small full config: {checked} rows of prompt {p} checked, {excused} near-ties excused")
    assert checked >= m * S // 2 and excused <= checked // 5

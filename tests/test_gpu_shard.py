"""Prompt-shard equivalence on one GPU: the data-parallel split of a batch
(Sec. 4.2.1 prices a batch as the maximum over its data-parallel groups).
A batch of P prompts is run whole, then as two shards [0, P/2) and
[P/2, P) in two contexts one after the other, each shard with
traj_base = first prompt * m.  Every trajectory must draw the same random
numbers in its shard as in the whole batch, so:

  * tiny fp32 model, free-running: the same tokens, lengths, statuses,
    completion steps and kept sets, and log-probs / entropies within the fp32
    bar (1e-5); with traj_base = 0 the second shard's tokens differ (the base
    is what makes them equal);
  * dense-small bf16 model, teacher-forced with one token table: the same
    schedule, statuses, lengths and kept sets, the GPU's own samples equal
    except where the two runs' logits differ by bf16 rounding near a tie
    (the GEMM and attention plans depend on the batch size, so low bits of
    the logits do), log-probs within the bf16 logit bar.
"""
import sys
from dataclasses import replace

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from workload import get_config, rollout_inputs
from workload.gen import teacher_forcing_tokens

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _run(model, run, prompts, forced, traj_base=0, tokens=None):
    """Rollout of prompts (P_run of them) on its own context; per local
    trajectory: taken tokens, own samples, log-probs, entropies; final
    scores, kept sets, completion steps."""
    from paper_2605_30859_amd import binding as B
    B.load_library()
    ro = B.Rollout(model, run, traj_base=traj_base)
    n = run.n_prompts * run.m
    pr = torch.from_numpy(np.ascontiguousarray(prompts.reshape(-1))).to(DEV)
    fl = torch.from_numpy(np.ascontiguousarray(forced).astype(np.int32)).to(DEV)
    hist = {key: [[] for _ in range(n)] for key in ("token", "sampled", "logprob", "entropy")}

    def force_fn(s):
        if tokens is None or s >= tokens.shape[1]:
            return None
        return torch.from_numpy(np.ascontiguousarray(tokens[:, s]).astype(np.int32)).to(DEV)

    def on_step(s, rows):
        h = {key: v.cpu().numpy() for key, v in rows.items()}
        for r, g in enumerate(h["traj"]):
            for key in hist:
                hist[key][int(g)].append(h[key][r])

    stats = ro.run_to_completion(pr, fl, on_step=on_step, force_fn=force_fn)
    ln, slp, mlp, st = [t.cpu().numpy() for t in ro.traj_scores()]
    out = dict(hist=hist, kept=ro.kept.cpu().numpy(), done=ro.done_step.cpu().numpy(), length=ln,
               sum_lp=slp, status=st, steps=stats["steps"])
    ro.close()
    return out


def _shards(name, tokens_steps=None, **run_over):
    model, run = get_config(name, **run_over)
    prompts, forced = rollout_inputs(model, run)
    P, m = run.n_prompts, run.m
    tokens = teacher_forcing_tokens(model, run, tokens_steps) if tokens_steps else None
    say(f"{name}: whole batch of {P} prompts")
    whole = _run(model, run, prompts, forced, 0, tokens)
    parts = []
    for a, b in ((0, P // 2), (P // 2, P)):
        say(f"{name}: shard [{a}, {b}), traj_base {a * m}")
        sub = replace(run, n_prompts=b - a)
        parts.append((a, _run(model, sub, prompts[a:b], forced[a * m:b * m], a * m,
                              None if tokens is None else tokens[a * m:b * m])))
    return model, run, prompts, forced, tokens, whole, parts


def _compare_schedule(run, whole, parts):
    m = run.m
    for a, part in parts:
        n = len(part["length"])
        sl = slice(a * m, a * m + n)
        assert np.array_equal(part["length"], whole["length"][sl])
        assert np.array_equal(part["status"], whole["status"][sl])
        assert np.array_equal(part["done"], whole["done"][a:a + len(part["done"])])
        assert np.array_equal(part["kept"] + a * m, whole["kept"][a:a + len(part["kept"])])


def test_tiny_shards_equal_whole_batch():
    model, run, prompts, forced, _, whole, parts = _shards("tiny")
    _compare_schedule(run, whole, parts)
    m = run.m
    worst = 0.0
    for a, part in parts:
        for j in range(len(part["length"])):
            g = a * m + j
            assert part["hist"]["token"][j] == whole["hist"]["token"][g], g
            assert part["hist"]["sampled"][j] == whole["hist"]["sampled"][g], g
            d = max(np.max(np.abs(np.subtract(part["hist"]["logprob"][j], whole["hist"]["logprob"][g]))),
                    np.max(np.abs(np.subtract(part["hist"]["entropy"][j], whole["hist"]["entropy"][g]))))
            worst = max(worst, float(d))
    say(f"tiny shards: tokens and schedule equal, worst score deviation {worst:.2e}")
    assert worst <= 1e-5
    # the base matters: the second shard run with traj_base 0 draws other numbers
    a, _ = parts[1]
    sub = replace(run, n_prompts=run.n_prompts - a)
    wrong = _run(model, sub, prompts[a:], forced[a * m:], 0)
    differ = sum(wrong["hist"]["sampled"][j] != whole["hist"]["sampled"][a * m + j]
                 for j in range(len(wrong["length"])))
    assert differ > 0


def test_dense_small_shards_equal_whole_batch():
    model, run, prompts, forced, tokens, whole, parts = _shards(
        "dense-small", tokens_steps=40, n_prompts=4, prompt_len=64, cap=40, len_median=16.0, kv_pool_gb=0.0)
    _compare_schedule(run, whole, parts)
    m = run.m
    rows = same = 0
    worst = 0.0
    for a, part in parts:
        for j in range(len(part["length"])):
            g = a * m + j
            assert part["hist"]["token"][j] == whole["hist"]["token"][g], g
            ps, ws = np.array(part["hist"]["sampled"][j]), np.array(whole["hist"]["sampled"][g])
            rows += len(ps)
            same += int((ps == ws).sum())
            worst = max(worst, float(np.max(np.abs(np.subtract(part["hist"]["logprob"][j],
                                                                whole["hist"]["logprob"][g])))))
    say(f"dense-small shards: schedule, taken tokens and kept sets equal; own samples equal on "
        f"{same} of {rows} rows; worst log-prob deviation {worst:.2e}")
    assert same >= 0.97 * rows and worst <= 0.25

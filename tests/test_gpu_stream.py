"""Token-chunk streaming (Sec. 4.3.2, producer side) on the GPU against the
oracle: dispatch steps, descriptors (trajectory, start, count, final status)
and token payloads, per step of a teacher-forced tiny rollout; the
per-trajectory concatenation on a bf16 dense-small rollout; the capacity
error leaves the state unchanged."""
from dataclasses import replace

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import model as OM
from oracle.rollout import rollout, schedule_only
from oracle.streaming import stream_chunks
from workload import get_config, rollout_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _b():
    from paper_2605_30859_amd import binding
    binding.load_library()
    return binding


def _stream_run(model, run, prompts, forced, threshold, force_tokens=None, out_cap=None):
    B = _b()
    ro = B.Rollout(model, run, flags=B.FLAG_STREAM)
    pr = torch.from_numpy(np.ascontiguousarray(prompts.reshape(-1))).to(DEV)
    fl = torch.from_numpy(forced.astype(np.int32)).to(DEV)
    disp, emitted = [], {}

    def force(s):
        if force_tokens is None:
            return None
        f = np.full(run.n_prompts * run.m, -1, dtype=np.int32)
        for g, toks in force_tokens.items():
            if s < len(toks):
                f[g] = toks[s]
        return torch.from_numpy(f).to(DEV)

    def record(rows):
        for g, t in zip(rows["traj"].cpu().numpy(), rows["token"].cpu().numpy()):
            emitted.setdefault(int(g), []).append(int(t))

    record(ro.darts_prefill(pr, fl, force(0)))
    ro.darts_select_and_prune()
    step = 1
    while True:
        r = ro.stream_chunks(threshold, flush=ro.n_done == run.n_prompts, out_cap=out_cap)
        if r is not None:
            disp.append((step, r))
        if ro.n_done == run.n_prompts:
            break
        record(ro.darts_decode_step(force(step)))
        ro.darts_select_and_prune()
        step += 1
    ro.close()
    return disp, emitted, step


@pytest.mark.parametrize("threshold", [1, 16, 100, 10 ** 9])
def test_tiny_stream_matches_oracle(threshold):
    model, run = get_config("tiny")
    prompts, forced = rollout_inputs(model, run)
    W = OM.init_weights(model)
    ref = rollout(model, W, prompts, forced, run.m, run.k, run.cap, run.sample_seed)
    exp = stream_chunks(ref.length, ref.tokens, ref.logprobs, ref.status, ref.steps, threshold)
    got, _, steps = _stream_run(model, run, prompts, forced, threshold, force_tokens=ref.tokens)
    assert steps == ref.steps
    assert [s for s, _ in got] == [s for s, _ in exp]
    for (s, (desc, tok, lp)), (_, chunks) in zip(got, exp):
        assert len(desc) == len(chunks)
        o = 0
        for (g, start, cnt, fin), (eg, estart, etk, elp, efin) in zip(desc, chunks):
            assert (g, start, cnt, fin) == (eg, estart, len(etk), efin)
            assert list(tok[o:o + cnt]) == etk
            assert np.allclose(lp[o:o + cnt], elp, atol=1e-5, rtol=0)
            o += cnt
        assert o == len(tok)


def test_dense_small_concatenation():
    """bf16 dense-small (cap 512): per trajectory, the chunks concatenate to
    exactly the tokens the decode steps emitted; dispatch steps and
    descriptors follow the oracle's rule on the same schedule."""
    model, run = get_config("dense-small")
    run = replace(run, cap=512)
    prompts, forced = rollout_inputs(model, run)
    got, emitted, steps = _stream_run(model, run, prompts, forced, threshold=4096)
    cat = {}
    for _, (desc, tok, lp) in got:
        o = 0
        for g, start, cnt, fin in desc:
            assert start == len(cat.get(int(g), []))
            cat.setdefault(int(g), []).extend(int(t) for t in tok[o:o + cnt])
            o += cnt
    assert cat == emitted
    s = schedule_only(forced, run.n_prompts, run.m, run.k, run.cap, run.prompt_len,
                      mean_lp=np.zeros(run.n_prompts * run.m, np.float32))
    length = {g: s["length"][g] for g in range(run.n_prompts * run.m)}
    assert {g: len(v) for g, v in cat.items()} == length
    dummy = {g: [0] * length[g] for g in length}
    exp = stream_chunks(length, dummy, dummy, {g: s["status"][g] for g in length}, s["steps"], 4096)
    assert [st for st, _ in got] == [st for st, _ in exp]
    for (_, (desc, _, _)), (_, chunks) in zip(got, exp):
        assert [tuple(int(v) for v in d[:3]) for d in desc] == [(g, a, len(t)) for g, a, t, _, _ in chunks]


def test_capacity_error_keeps_state():
    B = _b()
    model, run = get_config("tiny")
    prompts, forced = rollout_inputs(model, run)
    ro = B.Rollout(model, run, flags=B.FLAG_STREAM)
    pr = torch.from_numpy(np.ascontiguousarray(prompts.reshape(-1))).to(DEV)
    fl = torch.from_numpy(forced.astype(np.int32)).to(DEV)
    ro.darts_prefill(pr, fl)
    ro.darts_select_and_prune()
    for _ in range(3):
        ro.darts_decode_step()
        ro.darts_select_and_prune()
    n = run.n_prompts * run.m
    with pytest.raises(B.DartsError) as e:
        ro.stream_chunks(1, out_cap=5)
    assert e.value.status == B.DARTS_ENOMEM
    desc, tok, lp = ro.stream_chunks(1)
    assert len(desc) == n and (desc[:, 1] == 0).all() and (desc[:, 2] == 4).all()
    assert len(tok) == 4 * n
    ro.close()
    plain = B.Rollout(model, run)
    with pytest.raises(B.DartsError) as e:
        plain.stream_chunks(1)
    assert e.value.status == B.DARTS_ESTATE
    plain.close()

"""Caller-provided weights (darts_model_cfg.weights).  The oracle's own
tensors (generated in float64 from the seed by the oracle, rounded to bf16 for
bf16 models) are uploaded in the order and row-major layout the header
documents and given to a context whose weight_seed is different.  Its rollout
must equal, bit for bit, that of a context that generates the same weights
from the original seed on the device: tokens, own samples, log-probs,
entropies and kept sets at every step.  So the copy into the context's layout
(fused QKV rows, gate/up rows interleaved for the SwiGLU epilogue, expert
tensors, the padded router) is exact, for a dense and a mixture-of-experts
model; the caller's tensors can be freed once the context exists."""
import sys
from dataclasses import replace

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import model as OM
from workload import get_config, rollout_inputs
from workload.configs import ModelCfg

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _weights_on_device(model, W):
    dt = torch.bfloat16 if model.dtype == "bf16" else torch.float32
    up = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(dt).contiguous()
    ts = [up(W.embed), up(W.lm_head)]
    for lw in W.layers:
        ts += [up(lw.wq), up(lw.wk), up(lw.wv), up(lw.wo)]
        if model.n_experts:
            ts += [up(lw.router), up(lw.egate), up(lw.eup), up(lw.edown)]
        else:
            ts += [up(lw.wgate), up(lw.wup), up(lw.wdown)]
    return ts


def _run(model, run, prompts, forced, weights=None):
    from paper_2605_30859_amd import binding as B
    B.load_library()
    ro = B.Rollout(model, run, weights=weights)
    if weights is not None:
        del weights[:]                  # the context holds its own copy
        torch.cuda.synchronize()
    pr = torch.from_numpy(np.ascontiguousarray(prompts.reshape(-1))).to(DEV)
    fl = torch.from_numpy(np.ascontiguousarray(forced).astype(np.int32)).to(DEV)
    steps = []
    ro.run_to_completion(pr, fl, on_step=lambda s, rows: steps.append(
        {k: v.cpu().numpy().copy() for k, v in rows.items()}))
    out = dict(steps=steps, kept=ro.kept.cpu().numpy())
    ro.close()
    return out


def _same(a, b):
    assert len(a["steps"]) == len(b["steps"])
    for s, (x, y) in enumerate(zip(a["steps"], b["steps"])):
        for key in ("traj", "token", "sampled", "logprob", "entropy"):
            assert np.array_equal(x[key].view(np.uint32) if x[key].dtype == np.float32 else x[key],
                                  y[key].view(np.uint32) if y[key].dtype == np.float32 else y[key]), (s, key)
    assert np.array_equal(a["kept"], b["kept"])


def _check(model, run, label, check_seed_matters=False):
    prompts, forced = rollout_inputs(model, run)
    say(f"{label}: oracle weights")
    W = OM.init_weights(model)
    say(f"{label}: GPU, weights generated from the seed")
    ref = _run(model, run, prompts, forced)
    other = replace(model, weight_seed=model.weight_seed + 1000003)
    say(f"{label}: GPU, the oracle's weights passed in, other seed")
    got = _run(other, run, prompts, forced, _weights_on_device(model, W))
    _same(ref, got)
    say(f"{label}: {len(ref['steps'])} steps bit-identical")
    if check_seed_matters:
        alt = _run(other, run, prompts, forced)
        assert any(not np.array_equal(x["sampled"], y["sampled"]) for x, y in zip(ref["steps"], alt["steps"]))


def test_caller_weights_dense_fp32():
    model, run = get_config("tiny")
    _check(model, run, "tiny", check_seed_matters=True)


def test_caller_weights_moe_bf16():
    model = ModelCfg("moe-small", 2, 256, 4, 2, 64, 0, 512, "bf16", 21, rope_theta=1e6,
                     n_experts=16, top_k=4, expert_ffn=256)
    _, run = get_config("qwen3-30b-a3b")
    run = replace(run, n_prompts=2, prompt_len=32, m=8, k=4, cap=24, len_median=10.0, len_tail=False,
                  kv_pool_gb=0.0)
    _check(model, run, "moe-small")


def test_caller_weight_outside_device_memory_rejected():
    """An entry that is not inside a device allocation (here a host buffer)
    is rejected with DARTS_EINVAL before anything is copied."""
    import ctypes
    from paper_2605_30859_amd import binding as B
    lib = B.load_library()
    model, run = get_config("tiny")
    W = OM.init_weights(model)
    ts = _weights_on_device(model, W)
    host = np.zeros(ts[5].numel(), dtype=np.float32)
    arr = B.weight_pointer_array(ts)
    arr[5] = host.ctypes.data
    mc = B.model_cfg_struct(model, arr)
    rc = B.run_cfg_struct(run, torch.cuda.current_stream().cuda_stream)
    ctx = ctypes.c_void_p()
    st = lib.darts_init(ctypes.byref(mc), run.m, run.k, ctypes.byref(rc), ctypes.byref(ctx))
    assert st == B.DARTS_EINVAL and not ctx.value
    # the same tensors with the device entry back in place are accepted
    arr[5] = ts[5].data_ptr()
    mc = B.model_cfg_struct(model, arr)
    assert lib.darts_init(ctypes.byref(mc), run.m, run.k, ctypes.byref(rc), ctypes.byref(ctx)) == B.DARTS_OK
    assert lib.darts_destroy(ctx) == B.DARTS_OK

"""Pins for the layer-major teacher-forced oracle (oracle/forced.py) and the
helpers it uses: logits equal oracle.model.forward_sequence over each
trajectory's whole token sequence (which is itself pinned to a PyTorch
forward), the MoE routing it reports is the routing that forward applies, the
per-expert MoE evaluation equals the per-row one, row-wise and parallel
weight generation equal the plain generator, and the teacher-forcing window
follows the termination rule."""
import multiprocessing as mp

import numpy as np
import pytest

from oracle import model as M
from oracle.forced import forced_forward, taken_tokens
from workload.configs import ModelCfg


def cfg_dense():
    return ModelCfg("t", 2, 64, 4, 2, 16, 96, 97 * 4, "f32", 5)


def cfg_moe():
    return ModelCfg("t", 2, 64, 4, 1, 16, 0, 64, "bf16", 6, rope_theta=1e6, n_experts=8, top_k=3,
                    expert_ffn=32)


def _reference(cfg, W, prompts, traj_prompt, consumed):
    """forward_sequence over prompt + consumed tokens: logits for generated
    token s (s = 0 .. S-1) at position Lp - 1 + s, and per-layer margins."""
    Lp = prompts.shape[1]
    out, mars = [], []
    for t, p in enumerate(traj_prompt):
        seq = np.concatenate([prompts[p], consumed[t]])
        mar = []
        lg, _ = M.forward_sequence(cfg, W, seq, margins=mar)
        out.append(lg[Lp - 1:])
        mars.append(mar)
    return np.stack(out), mars


@pytest.mark.parametrize("make", [cfg_dense, cfg_moe])
def test_forced_forward_equals_sequence_forward(make):
    cfg = make()
    W = M.init_weights(cfg)
    rng = np.random.default_rng(3)
    Lp, S = 12, 6
    prompts = rng.integers(0, cfg.vocab, (2, Lp))
    traj_prompt = np.array([0, 1, 1, 0, 1])
    consumed = rng.integers(0, cfg.vocab, (len(traj_prompt), S - 1))
    routing = {}
    last, dec = forced_forward(cfg, prompts, traj_prompt, consumed, lambda l: W.layers[l],
                               lambda tk: W.embed[np.asarray(tk)], routing=routing)
    ref, mars = _reference(cfg, W, prompts, traj_prompt, consumed)
    for t, p in enumerate(traj_prompt):
        np.testing.assert_allclose(last[p] @ W.lm_head.T, ref[t, 0], rtol=0, atol=1e-11)
        np.testing.assert_allclose(dec[t] @ W.lm_head.T, ref[t, 1:], rtol=0, atol=1e-11)
    if cfg.n_experts:
        n_pre = prompts.size
        ids, pp, mg = routing["ids"], routing["p"], routing["margin"]
        assert ids.shape == (n_pre + len(traj_prompt) * (S - 1), cfg.n_layers, cfg.top_k)
        for t, p in enumerate(traj_prompt):
            for l in range(cfg.n_layers):
                # prompt rows of prompt p, then this trajectory's decode rows
                rows = np.concatenate([np.arange(p * Lp, (p + 1) * Lp),
                                       n_pre + t * (S - 1) + np.arange(S - 1)])
                np.testing.assert_allclose(mg[rows, l], mars[t][l], rtol=0, atol=1e-13)
        # probabilities at the ids are in rank order and the margin is the k/k+1 gap
        assert (np.diff(pp, axis=-1) <= 0).all() and (mg >= 0).all() and (mg <= pp[..., -1]).all()


def test_moe_by_expert_equals_per_row():
    cfg = cfg_moe()
    W = M.init_weights(cfg)
    h = np.random.default_rng(4).standard_normal((37, cfg.d_model))
    out, ids, pid, mar = M.moe_ffn_by_expert(cfg, W.layers[1], h)
    mars = []
    ref = M.ffn(cfg, W.layers[1], h, margins=mars)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-13)
    np.testing.assert_array_equal(mar, mars[0])
    i2, w2, p2 = M.moe_route(cfg, W.layers[1].router, h)
    np.testing.assert_array_equal(ids, i2)
    np.testing.assert_array_equal(pid, np.take_along_axis(p2, i2, axis=-1))


def test_init_rows_and_parallel_init_equal_plain():
    full = M.init_tensor(9, M.T_EMBED, 0, 50, 24, 1, "bf16")
    rows = [0, 7, 49, 7]
    np.testing.assert_array_equal(M.init_rows(9, M.T_EMBED, 0, rows, 24, 1, "bf16"), full[rows])
    with mp.get_context("fork").Pool(2) as pool:
        par = M.init_tensor(9, M.T_EMBED, 0, 50, 24, 1, "bf16", chunk=100, pool=pool)
    np.testing.assert_array_equal(par, full)


def test_taken_tokens_window():
    tok = np.arange(20).reshape(4, 5) + 100
    # window of 5 tokens, cap 4: d = 3 ends with eos as token index 2; d = 9
    # and d = 5 exceed the cap and are truncated after 4 tokens (no eos);
    # d = 2 ends with eos as token index 1
    taken, n = taken_tokens([3, 9, 2, 5], tok, cap=4, eos=7)
    assert list(n) == [3, 4, 2, 4]
    assert list(taken[0]) == [100, 101, 7, 103, 104]
    assert list(taken[1]) == list(tok[1])
    assert list(taken[2]) == [110, 7, 112, 113, 114]
    assert list(taken[3]) == list(tok[3])
    # a cap beyond the window: d = 9 runs through it, d = 5 ends at its last token
    taken, n = taken_tokens([9, 5], tok[:2], cap=100, eos=7)
    assert list(n) == [5, 5] and taken[1, 4] == 7 and list(taken[0]) == list(tok[0])

"""Pins for the oracle decoder: a PyTorch CPU float64 forward built from the
same weights with library routines (scaled_dot_product_attention, rms_norm,
silu), closed-form special cases, and the weight-init statistics."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

from oracle import model as M
from workload.configs import ModelCfg


def small_cfg(**kw):
    base = dict(name="t", n_layers=2, d_model=64, n_q_heads=4, n_kv_heads=2, head_dim=16,
                ffn_dim=96, vocab=97, dtype="f32", weight_seed=11)
    base.update(kw)
    return ModelCfg(**base)


def torch_forward(cfg, W, tokens):
    """Independent forward with torch library ops (causal SDPA with GQA, rms_norm)."""
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(torch.float64)
    n = len(tokens)
    hq, hkv, hd = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    x = t(W.embed)[torch.as_tensor(tokens)]
    pos = torch.arange(n, dtype=torch.float64)
    half = hd // 2
    inv = cfg.rope_theta ** (-2.0 * torch.arange(half, dtype=torch.float64) / hd)
    ang = pos[:, None] * inv[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)            # e^{i p theta}

    def rope(v):          # v: [n, H, hd] as complex pairs (a_i + i a_{i+half})
        c = torch.complex(v[..., :half], v[..., half:]) * rot[:, None, :]
        return torch.cat([c.real, c.imag], dim=-1)

    for lw in W.layers:
        h = Fn.rms_norm(x, (cfg.d_model,), eps=cfg.rms_eps)
        q = rope((h @ t(lw.wq).T).view(n, hq, hd)).transpose(0, 1)
        k = rope((h @ t(lw.wk).T).view(n, hkv, hd)).transpose(0, 1)
        v = (h @ t(lw.wv).T).view(n, hkv, hd).transpose(0, 1)
        o = Fn.scaled_dot_product_attention(q[None], k[None], v[None], is_causal=True,
                                            enable_gqa=True)[0]
        x = x + o.transpose(0, 1).reshape(n, hq * hd) @ t(lw.wo).T
        h = Fn.rms_norm(x, (cfg.d_model,), eps=cfg.rms_eps)
        if cfg.n_experts == 0:
            x = x + (Fn.silu(h @ t(lw.wgate).T) * (h @ t(lw.wup).T)) @ t(lw.wdown).T
        else:
            pr = torch.softmax(h @ t(lw.router).T, dim=-1)
            top = torch.topk(pr, cfg.top_k, dim=-1)
            wts = top.values / top.values.sum(-1, keepdim=True)
            out = torch.zeros_like(x)
            for r in range(n):
                for j in range(cfg.top_k):
                    e = int(top.indices[r, j])
                    a = Fn.silu(t(lw.egate[e]) @ h[r]) * (t(lw.eup[e]) @ h[r])
                    out[r] += wts[r, j] * (t(lw.edown[e]) @ a)
            x = x + out
    return (Fn.rms_norm(x, (cfg.d_model,), eps=cfg.rms_eps) @ t(W.lm_head).T).numpy()


@pytest.mark.parametrize("kw", [dict(), dict(n_kv_heads=4), dict(n_kv_heads=1),
                                dict(dtype="bf16"), dict(rope_theta=1e6)])
def test_forward_matches_torch(kw):
    cfg = small_cfg(**kw)
    W = M.init_weights(cfg)
    toks = np.random.default_rng(0).integers(0, cfg.vocab, 23)
    ref = torch_forward(cfg, W, toks)
    got, _ = M.forward_sequence(cfg, W, toks)
    assert np.max(np.abs(got - ref)) < 1e-10 * max(1.0, np.max(np.abs(ref)))


def test_moe_forward_matches_torch():
    cfg = small_cfg(ffn_dim=0, n_experts=8, top_k=2, expert_ffn=24)
    W = M.init_weights(cfg)
    toks = np.random.default_rng(1).integers(0, cfg.vocab, 9)
    ref = torch_forward(cfg, W, toks)
    got, _ = M.forward_sequence(cfg, W, toks)
    assert np.max(np.abs(got - ref)) < 1e-10 * max(1.0, np.max(np.abs(ref)))


def test_incremental_decode_equals_full_sequence():
    cfg = small_cfg()
    W = M.init_weights(cfg)
    toks = np.random.default_rng(2).integers(0, cfg.vocab, 12)
    full, _ = M.forward_sequence(cfg, W, toks)
    lg, cache = M.forward_sequence(cfg, W, toks[:8])
    caches = [(c[0][None], c[1][None]) for c in cache]
    for p in range(8, 12):
        lgs, caches = M.decode_batch(cfg, W, [toks[p]], caches)
        assert np.max(np.abs(lgs[0] - full[p])) < 1e-11


def test_rope_position_zero_is_identity_and_preserves_norm():
    x = np.random.default_rng(3).normal(size=(5, 3, 16))
    assert np.array_equal(M.rope(x, 0, 1e4), x)
    y = M.rope(x, 37, 1e4)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), atol=1e-12)
    # relative position: <R_p q, R_r k> depends only on p - r
    q, k = x[0, 0], x[1, 0]
    a = M.rope(q[None, None], 10, 1e4)[0, 0] @ M.rope(k[None, None], 4, 1e4)[0, 0]
    b = M.rope(q[None, None], 26, 1e4)[0, 0] @ M.rope(k[None, None], 20, 1e4)[0, 0]
    assert abs(a - b) < 1e-12


def test_attention_special_cases():
    rng = np.random.default_rng(4)
    q = rng.normal(size=(4, 8))
    K = rng.normal(size=(1, 2, 8))
    V = rng.normal(size=(1, 2, 8))
    o = M.attention(q, K, V, 2)
    assert np.allclose(o[0], V[0, 0]) and np.allclose(o[3], V[0, 1])
    K = np.zeros((5, 1, 8))
    V = rng.normal(size=(5, 1, 8))
    o = M.attention(q[:1], K, V, 1)
    assert np.allclose(o[0], V[:, 0].mean(0))
    # GQA == MHA with replicated kv heads
    K = rng.normal(size=(6, 2, 8))
    V = rng.normal(size=(6, 2, 8))
    a = M.attention(q, K, V, 2)
    b = M.attention(q, np.repeat(K, 2, axis=1), np.repeat(V, 2, axis=1), 4)
    assert np.allclose(a, b, atol=1e-14)


def test_zeroed_blocks_give_lm_head_of_normalised_embedding():
    cfg = small_cfg(n_layers=1)
    W = M.init_weights(cfg)
    W.layers[0].wo[:] = 0
    W.layers[0].wdown[:] = 0
    toks = [5, 9, 11]
    got, _ = M.forward_sequence(cfg, W, toks)
    e = W.embed[toks]
    ref = (e / np.sqrt((e * e).mean(-1, keepdims=True) + cfg.rms_eps)) @ W.lm_head.T
    assert np.allclose(got, ref, atol=1e-12)


def test_weight_init_statistics_and_grid():
    w = M.init_tensor(5, M.T_WQ, 3, 256, 512, 512, "f32")
    assert abs(w.var() * 512 - 1.0) < 0.02      # variance 1/fan_in
    assert abs(w.mean()) < 2e-3
    a = np.float32(math.sqrt(3.0 / 512))
    v = (w / float(a))                               # back onto the (-1,1) grid (approx.)
    assert np.max(np.abs(v)) < 1.0 + 1e-6
    b = M.init_tensor(5, M.T_WQ, 3, 256, 512, 512, "bf16")
    bits = b.astype(np.float32).view(np.uint32)
    assert np.all(bits & 0xFFFF == 0)
    assert np.max(np.abs(b - w)) <= np.max(np.abs(w)) * 2 ** -8
    # different layers / tensors draw different values
    assert not np.array_equal(w, M.init_tensor(5, M.T_WQ, 4, 256, 512, 512, "f32"))
    assert not np.array_equal(w, M.init_tensor(5, M.T_WK, 3, 256, 512, 512, "f32"))


def test_round_bf16_nearest_even():
    x = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20, -2.5], dtype=np.float32)
    r = M.round_bf16(x)
    assert r[0] == 1.0 and r[1] == 1.0 + 4 * 2 ** -8 and r[2] == 1.0 + 2 * 2 ** -8 and r[3] == -2.5


def test_moe_route_ties_lower_id():
    cfg = small_cfg(ffn_dim=0, n_experts=6, top_k=2, expert_ffn=4)
    router = np.zeros((6, 64))
    router[4, 0] = 1.0
    h = np.zeros((1, 64))
    h[0, 0] = 1.0
    ids, w, p = M.moe_route(cfg, router, h)
    assert list(ids[0]) == [4, 0]
    assert abs(w[0].sum() - 1.0) < 1e-15

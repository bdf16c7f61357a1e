"""Random-init pre-norm decoder (dense SwiGLU or top-k MoE), float64 forward.

The paper does not describe its models' internals (it trains Qwen checkpoints
inside its rollout engine); the workloads specify Qwen-shaped decoders with
random initialisation.  The definitions used here:

Weights (logical layout [out][in], element index idx = o*in + i):
    word  = Philox(key=weight_seed, counter=(idx>>2, tensor_id, layer, TAG_WEIGHT)) word idx&3
    v     = ((word >> 8) | 1) * 2^-23 - 1                    (exact float32 in (-1, 1))
    w     = fl32(v * a),  a = fl32(sqrt(3 / fan_in))          (variance 1/fan_in)
    bf16 models round w to bfloat16 (nearest even) before any use.
Embedding uses a = fl32(sqrt(3)).  RMSNorm gains are 1, there are no biases,
the LM head is untied.

Forward, per token at position p:
    x = E[token]
    per layer:
        h = x / sqrt(mean(x^2) + eps)
        q, k, v = Wq h, Wk h, Wv h;   RoPE (rotate-half) on q and k:
            theta_i = base^(-2i/hd),  (a_i, a_{i+hd/2}) <- (a_i c - a_{i+hd/2} s, a_{i+hd/2} c + a_i s)
        attention per q head h, kv head floor(h * Hkv / Hq):
            softmax_j(q . k_j / sqrt(hd)) over all positions j <= p,  o = sum_j p_j v_j
        x = x + Wo o
        h = x / sqrt(mean(x^2) + eps)
        dense:  x = x + Wdown (silu(Wgate h) * (Wup h))
        MoE:    r = softmax(Wrouter h); top-k experts (ties -> lower id);
                weights renormalised over the k; x = x + sum_e w_e Wdown_e(silu(Wgate_e h) * (Wup_e h))
    logits = Wlm (x / sqrt(mean(x^2) + eps))

Pins: PyTorch CPU float64 forward built from the same weights (library check),
and special cases: RoPE at position 0 is the identity; attention over a single
key returns that value; GQA equals MHA with kv heads replicated; with
attention and FFN output projections zeroed the logits equal the LM head
applied to the normalised embedding (tests/test_oracle_model.py).
"""
from dataclasses import dataclass
import math

import numpy as np

from .philox import philox_range

TAG_WEIGHT = 1
T_EMBED, T_WQ, T_WK, T_WV, T_WO, T_WGATE, T_WUP, T_WDOWN, T_LM = range(9)
T_ROUTER, T_EGATE, T_EUP, T_EDOWN = 9, 10, 11, 12


def round_bf16(x32: np.ndarray) -> np.ndarray:
    """float32 -> nearest-even bfloat16 value, returned as float32."""
    b = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (b >> np.uint64(16)) & np.uint64(1)
    r = ((b + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    return r.astype(np.uint32).view(np.float32)


def _weight_values(args):
    """Elements [start, start + n) of one weight tensor, float32 (exact)."""
    start, n, tensor_id, layer, seed, fan_in, dtype = args
    a = np.float32(math.sqrt(3.0 / fan_in))
    w = philox_range(start, n, tensor_id, layer, TAG_WEIGHT, seed)
    k = ((w >> np.uint32(8)) | np.uint32(1)).astype(np.float32)
    v = (k * np.float32(2.0 ** -23) - np.float32(1.0)).astype(np.float32)
    x = (v * a).astype(np.float32)
    if dtype == "bf16":
        x = round_bf16(x)
    return x


def init_tensor(seed, tensor_id, layer, n_out, n_in, fan_in, dtype, chunk=1 << 24, pool=None):
    """Generate one weight tensor [n_out, n_in] as float64 (values exact in the model dtype).
    ``pool``: an optional multiprocessing pool that generates the chunks in parallel
    (the same elements; only the wall time changes)."""
    total = n_out * n_in
    out = np.empty(total, dtype=np.float64)
    jobs = [(s, min(total, s + chunk) - s, tensor_id, layer, seed, fan_in, dtype)
            for s in range(0, total, chunk)]
    parts = pool.imap(_weight_values, jobs) if pool is not None else map(_weight_values, jobs)
    for (s, n, *_), x in zip(jobs, parts):
        out[s:s + n] = x
    return out.reshape(n_out, n_in)


def init_rows(seed, tensor_id, layer, rows, n_in, fan_in, dtype):
    """Rows ``rows`` of the tensor init_tensor would generate, [len(rows), n_in]
    float64 (element (r, i) is element r * n_in + i of the tensor); n_in % 4 == 0."""
    assert n_in % 4 == 0
    rows = np.asarray(rows, dtype=np.int64).reshape(-1)
    out = np.empty((len(rows), n_in), dtype=np.float64)
    for j, r in enumerate(rows):
        out[j] = _weight_values((int(r) * n_in, n_in, tensor_id, layer, seed, fan_in, dtype))
    return out


@dataclass
class LayerW:
    wq: np.ndarray
    wk: np.ndarray
    wv: np.ndarray
    wo: np.ndarray
    wgate: np.ndarray = None
    wup: np.ndarray = None
    wdown: np.ndarray = None
    router: np.ndarray = None
    egate: np.ndarray = None     # [E, Fe, d]
    eup: np.ndarray = None       # [E, Fe, d]
    edown: np.ndarray = None     # [E, d, Fe]


def init_layer(cfg, layer, pool=None):
    s, d, dt = cfg.weight_seed, cfg.d_model, cfg.dtype
    hq, hkv, hd = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    it = lambda *a: init_tensor(*a, pool=pool)
    lw = LayerW(
        wq=it(s, T_WQ, layer, hq * hd, d, d, dt),
        wk=it(s, T_WK, layer, hkv * hd, d, d, dt),
        wv=it(s, T_WV, layer, hkv * hd, d, d, dt),
        wo=it(s, T_WO, layer, d, hq * hd, hq * hd, dt),
    )
    if cfg.n_experts:
        E, Fe = cfg.n_experts, cfg.expert_ffn
        lw.router = it(s, T_ROUTER, layer, E, d, d, dt)
        lw.egate = it(s, T_EGATE, layer, E * Fe, d, d, dt).reshape(E, Fe, d)
        lw.eup = it(s, T_EUP, layer, E * Fe, d, d, dt).reshape(E, Fe, d)
        lw.edown = it(s, T_EDOWN, layer, E * d, Fe, Fe, dt).reshape(E, d, Fe)
    else:
        F = cfg.ffn_dim
        lw.wgate = it(s, T_WGATE, layer, F, d, d, dt)
        lw.wup = it(s, T_WUP, layer, F, d, d, dt)
        lw.wdown = it(s, T_WDOWN, layer, d, F, F, dt)
    return lw


@dataclass
class Weights:
    embed: np.ndarray
    layers: list
    lm_head: np.ndarray


def init_weights(cfg):
    s, d, V, dt = cfg.weight_seed, cfg.d_model, cfg.vocab, cfg.dtype
    return Weights(embed=init_tensor(s, T_EMBED, 0, V, d, 1, dt),
                   layers=[init_layer(cfg, l) for l in range(cfg.n_layers)],
                   lm_head=init_tensor(s, T_LM, 0, V, d, d, dt))


def rmsnorm(x, eps):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def rope(x, pos, base):
    """Rotate-half RoPE.  x: [..., n_heads, hd]; pos: broadcastable to x[..., 0, 0]."""
    hd = x.shape[-1]
    half = hd // 2
    inv = base ** (-2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = np.asarray(pos, dtype=np.float64)[..., None, None] * inv
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def silu(x):
    return x / (1.0 + np.exp(-x))


def moe_route(cfg, router_w, h):
    """Top-k expert ids (ascending rank order) and renormalised weights for rows of h."""
    logits = h @ router_w.T
    z = logits - logits.max(axis=-1, keepdims=True)
    p = np.exp(z)
    p /= p.sum(axis=-1, keepdims=True)
    # stable sort on -p: equal probabilities keep ascending expert id
    order = np.argsort(-p, axis=-1, kind="stable")[:, :cfg.top_k]
    w = np.take_along_axis(p, order, axis=-1)
    w = w / w.sum(axis=-1, keepdims=True)
    return order, w, p


def route_margin(cfg, p):
    """Per row: probability gap between the k-th and (k+1)-th expert (how far
    the top-k decision is from a tie)."""
    srt = -np.sort(-p, axis=-1)
    if cfg.top_k >= p.shape[-1]:
        return np.full(p.shape[0], np.inf)
    return srt[:, cfg.top_k - 1] - srt[:, cfg.top_k]


def ffn(cfg, lw, h, margins=None):
    if cfg.n_experts == 0:
        return (silu(h @ lw.wgate.T) * (h @ lw.wup.T)) @ lw.wdown.T
    ids, w, p = moe_route(cfg, lw.router, h)
    if margins is not None:
        margins.append(route_margin(cfg, p))
    out = np.zeros_like(h)
    for r in range(h.shape[0]):
        for j in range(cfg.top_k):
            e = ids[r, j]
            a = silu(lw.egate[e] @ h[r]) * (lw.eup[e] @ h[r])
            out[r] += w[r, j] * (lw.edown[e] @ a)
    return out


def moe_ffn_by_expert(cfg, lw, h):
    """The MoE FFN of ``ffn`` for many rows at once: routing as in moe_route,
    y[r, j] = expert_{ids[r, j]}(h[r]) evaluated for all rows routed to an
    expert together (one matrix product per expert), then
    out[r] = sum_j w[r, j] y[r, j] in slot order j.
    Returns (out, ids [n, k], p at ids [n, k] (softmax probabilities before
    renormalisation), route_margin [n])."""
    ids, w, p = moe_route(cfg, lw.router, h)
    n, k = ids.shape
    y = np.empty((n, k, h.shape[1]))
    for e in np.unique(ids):
        rr, jj = np.nonzero(ids == e)
        a = silu(h[rr] @ lw.egate[e].T) * (h[rr] @ lw.eup[e].T)
        y[rr, jj] = a @ lw.edown[e].T
    out = np.zeros_like(h)
    for j in range(k):
        out += w[:, j:j + 1] * y[:, j]
    return out, ids, np.take_along_axis(p, ids, axis=-1), route_margin(cfg, p)


def attention(q, K, V, n_kv):
    """q: [Hq, hd]; K, V: [ctx, Hkv, hd] -> [Hq, hd].  Softmax(q k / sqrt(hd)) v."""
    hq, hd = q.shape
    out = np.empty_like(q)
    for h in range(hq):
        kh = (h * n_kv) // hq
        s = K[:, kh, :] @ q[h] / math.sqrt(hd)
        s = s - s.max()
        p = np.exp(s)
        p /= p.sum()
        out[h] = p @ V[:, kh, :]
    return out


def forward_sequence(cfg, W, tokens, cache=None, margins=None):
    """Causal forward over ``tokens`` appended after an optional cache.

    cache: list per layer of (K [ctx, Hkv, hd], V [ctx, Hkv, hd]) or None.
    Returns (logits [len(tokens), V], new cache).
    """
    hq, hkv, hd = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    n = len(tokens)
    start = 0 if cache is None else cache[0][0].shape[0]
    pos = np.arange(start, start + n)
    x = W.embed[np.asarray(tokens)]
    new_cache = []
    for l, lw in enumerate(W.layers):
        h = rmsnorm(x, cfg.rms_eps)
        q = rope((h @ lw.wq.T).reshape(n, hq, hd), pos, cfg.rope_theta)
        k = rope((h @ lw.wk.T).reshape(n, hkv, hd), pos, cfg.rope_theta)
        v = (h @ lw.wv.T).reshape(n, hkv, hd)
        if cache is not None:
            K = np.concatenate([cache[l][0], k], axis=0)
            V = np.concatenate([cache[l][1], v], axis=0)
        else:
            K, V = k, v
        new_cache.append((K, V))
        o = np.empty((n, hq, hd))
        for t in range(n):
            ctx = start + t + 1
            o[t] = attention(q[t], K[:ctx], V[:ctx], hkv)
        x = x + o.reshape(n, hq * hd) @ lw.wo.T
        h = rmsnorm(x, cfg.rms_eps)
        x = x + ffn(cfg, lw, h, margins)
    logits = rmsnorm(x, cfg.rms_eps) @ W.lm_head.T
    return logits, new_cache


def decode_batch(cfg, W, tokens, caches, margins=None):
    """One decode step for B sequences that all have the same cached length.

    tokens: [B]; caches: list per layer of (K [B, ctx, Hkv, hd], V [B, ctx, Hkv, hd]).
    margins: optional list; for MoE models one array [B] of routing margins
    per layer is appended.
    Returns (logits [B, V], caches extended by one position).
    """
    hq, hkv, hd = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    B = len(tokens)
    ctx0 = caches[0][0].shape[1]
    x = W.embed[np.asarray(tokens)]
    out_caches = []
    g = hq // hkv
    for l, lw in enumerate(W.layers):
        h = rmsnorm(x, cfg.rms_eps)
        q = rope((h @ lw.wq.T).reshape(B, hq, hd), ctx0, cfg.rope_theta)
        k = rope((h @ lw.wk.T).reshape(B, hkv, hd), ctx0, cfg.rope_theta)
        v = (h @ lw.wv.T).reshape(B, hkv, hd)
        K = np.concatenate([caches[l][0], k[:, None]], axis=1)
        V = np.concatenate([caches[l][1], v[:, None]], axis=1)
        out_caches.append((K, V))
        # scores [B, Hq, ctx]: q head h reads kv head h // g
        Kx = np.repeat(K, g, axis=2)             # [B, ctx, Hq, hd]
        Vx = np.repeat(V, g, axis=2)
        s = np.einsum("bhd,bchd->bhc", q, Kx) / math.sqrt(hd)
        s = s - s.max(axis=-1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=-1, keepdims=True)
        o = np.einsum("bhc,bchd->bhd", p, Vx)
        x = x + o.reshape(B, hq * hd) @ lw.wo.T
        h = rmsnorm(x, cfg.rms_eps)
        x = x + ffn(cfg, lw, h, margins)
    logits = rmsnorm(x, cfg.rms_eps) @ W.lm_head.T
    return logits, out_caches

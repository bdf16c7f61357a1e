"""Teacher-forced forward of a few prompts and their trajectories, one decoder
layer at a time (float64).  Test infrastructure: the parity reference for the
large configurations, whose weights (16-61 GB in the model dtype, four to
eight times that in float64) never have to be held at once.

Definition.  Prompt p has tokens prompts[p] (positions 0 .. Lp-1).  Trajectory
t extends prompt traj_prompt[t]; its generated token 0 is scored from the
prompt's last-position logits, and its decode step s >= 1 consumes
consumed[t, s-1] at position Lp + s - 1 and scores generated token s.  Every
row of the batch is the decoder of oracle.model applied to its own causal
context: a prompt position sees its prompt's earlier positions; decode step s
of trajectory t sees the whole prompt and the trajectory's own consumed
tokens up to and including position Lp + s - 1.  Because the consumed tokens
are known in advance (teacher forcing), the forward can run layer-major over
all rows: each layer's weights are generated, used for every row, and
dropped.  Nothing is blocked or reordered inside a row's arithmetic: the
same products, softmaxes and sums as oracle.model.forward_sequence over
prompt + consumed tokens, batched over rows.

Pinned by tests/test_oracle_forced.py: the logits equal forward_sequence over
each trajectory's full token sequence (dense and MoE models), and the routing
it reports equals the routing forward_sequence applies.
"""
import math

import numpy as np

from . import model as M


def forced_forward(cfg, prompts, traj_prompt, consumed, get_layer, embed_rows, routing=None):
    """Final-normalised hidden states of every scored row.

    prompts      [Ps, Lp] int token ids
    traj_prompt  [T] int, the prompt each trajectory extends
    consumed     [T, S-1] int, token consumed at decode step s = 1 .. S-1
    get_layer(l) -> oracle.model.LayerW of layer l
    embed_rows(tokens [n]) -> [n, d] embedding rows
    routing      None or a dict, filled for MoE models with per-row, per-layer
                 'ids' [R, L, k] (rank order), 'p' [R, L, k] (softmax
                 probabilities at those ids, before renormalisation) and
                 'margin' [R, L] (k-th minus (k+1)-th probability), rows R =
                 prefill rows (prompt-major, Ps*Lp) then decode rows
                 (trajectory-major, T*(S-1))

    Returns (h_prompt_last [Ps, d], h_decode [T, S-1, d]): RMSNorm of the
    final residual stream, the LM head's input for generated token 0 of each
    prompt's trajectories and for decode steps 1 .. S-1.
    """
    prompts = np.asarray(prompts)
    traj_prompt = np.asarray(traj_prompt)
    consumed = np.asarray(consumed).reshape(len(traj_prompt), -1)
    Ps, Lp = prompts.shape
    T, S1 = consumed.shape
    hq, hkv, hd, d = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_model
    eps, base = cfg.rms_eps, cfg.rope_theta
    scale = 1.0 / math.sqrt(hd)
    n_pre, n_dec = Ps * Lp, T * S1
    # residual stream of every row: prefill rows first, then decode rows
    x = np.concatenate([embed_rows(prompts.reshape(-1)), embed_rows(consumed.reshape(-1))], axis=0)
    pos = np.concatenate([np.tile(np.arange(Lp), Ps), np.tile(Lp + np.arange(S1), T)])
    if routing is not None and cfg.n_experts:
        R, k = n_pre + n_dec, cfg.top_k
        routing["ids"] = np.zeros((R, cfg.n_layers, k), dtype=np.int64)
        routing["p"] = np.zeros((R, cfg.n_layers, k))
        routing["margin"] = np.zeros((R, cfg.n_layers))
    causal_p = np.tril(np.ones((Lp, Lp), dtype=bool))
    # decode step i (0-based row of a trajectory) sees the prompt and decode keys 0..i
    causal_d = np.concatenate([np.ones((S1, Lp), dtype=bool), np.tril(np.ones((S1, S1), dtype=bool))], axis=1)

    def attend(q, K, V, mask):
        """q [n, hq, hd], K/V [c, hkv, hd], mask [n, c] -> [n, hq, hd]."""
        out = np.empty_like(q)
        # per-head operands as contiguous arrays, so the products go to BLAS
        Kt = [np.ascontiguousarray(K[:, j, :].T) for j in range(hkv)]
        Vh = [np.ascontiguousarray(V[:, j, :]) for j in range(hkv)]
        for h in range(hq):
            kh = (h * hkv) // hq
            s = (np.ascontiguousarray(q[:, h, :]) @ Kt[kh]) * scale
            s = np.where(mask, s, -np.inf)
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            out[:, h, :] = p @ Vh[kh]
        return out

    for l in range(cfg.n_layers):
        lw = get_layer(l)
        h = M.rmsnorm(x, eps)
        n = len(h)
        q = M.rope((h @ lw.wq.T).reshape(n, hq, hd), pos, base)
        kk = M.rope((h @ lw.wk.T).reshape(n, hkv, hd), pos, base)
        vv = (h @ lw.wv.T).reshape(n, hkv, hd)
        o = np.empty((n, hq, hd))
        qp, kp, vp = (a[:n_pre].reshape(Ps, Lp, *a.shape[1:]) for a in (q, kk, vv))
        qd, kd, vd = (a[n_pre:].reshape(T, S1, *a.shape[1:]) for a in (q, kk, vv))
        op = o[:n_pre].reshape(Ps, Lp, hq, hd)
        od = o[n_pre:].reshape(T, S1, hq, hd)
        for p in range(Ps):
            op[p] = attend(qp[p], kp[p], vp[p], causal_p)
        for t in range(T):
            p = traj_prompt[t]
            K = np.concatenate([kp[p], kd[t]], axis=0)
            V = np.concatenate([vp[p], vd[t]], axis=0)
            od[t] = attend(qd[t], K, V, causal_d)
        x = x + o.reshape(n, hq * hd) @ lw.wo.T
        h = M.rmsnorm(x, eps)
        if cfg.n_experts:
            y, ids, pid, mar = M.moe_ffn_by_expert(cfg, lw, h)
            if routing is not None:
                routing["ids"][:, l] = ids
                routing["p"][:, l] = pid
                routing["margin"][:, l] = mar
            x = x + y
        else:
            x = x + (M.silu(h @ lw.wgate.T) * (h @ lw.wup.T)) @ lw.wdown.T
        del lw
    hf = M.rmsnorm(x, eps)
    last = hf[:n_pre].reshape(Ps, Lp, d)[:, -1]
    return last, hf[n_pre:].reshape(T, S1, d)


def taken_tokens(forced_len, tokens, cap, eos):
    """The token each trajectory takes at generated index s = 0 .. S-1 under
    teacher forcing with ``tokens`` [T, S], and how many it generates in the
    window: the forced end-of-sequence (1-based count s + 1 = d <= cap) is
    taken instead of the forced token and ends the trajectory; d > cap
    truncates it at cap.  Returns (taken [T, S], n_gen [T])."""
    tokens = np.asarray(tokens)
    T, S = tokens.shape
    taken = tokens.copy()
    n_gen = np.full(T, S, dtype=np.int64)
    for t in range(T):
        d = int(forced_len[t])
        if d <= cap and d <= S:
            taken[t, d - 1] = eos
        n_gen[t] = min(S, d, cap)
    return taken, n_gen


def reference_values(cfg, run, prompts, forced, tokens, prompt_ids, n_steps, pool=None, n_idx=256,
                     idx_seed=2605, log=None):
    """The oracle's teacher-forced values for prompts ``prompt_ids`` of a batch
    and their m trajectories each (global ids g = i*m + j), for generated
    indices 0 .. n_steps-1, as a dict of arrays:

      traj [T], prompts [Ps], steps, tokens / taken [T, S] (forcing table and
      the tokens actually taken, the forced end-of-sequence included), n_gen [T]
      idx [n_idx] fixed vocabulary ids, logits_at_idx [T, S, n_idx]
      zmax, zabs, argmax, lse [T, S]: largest logit, largest |logit|, its id,
      log-sum-exp of the logits / T
      sampled, logprob, entropy, margin [T, S]: the Gumbel-max sample of
      (g, s), log-prob of the taken token, entropy, top-2 perturbed margin
      MoE: route_ids / route_p [R, L, k], route_margin [R, L] (forced_forward)

    Weights are generated layer by layer from the model's seed (``pool``: an
    optional multiprocessing pool for the generator and the sampler rows)."""
    from .sampler import sample_row, top2_margin
    say = log or (lambda *a: None)
    m, eos = run.m, cfg.vocab - 1
    prompt_ids = list(prompt_ids)
    traj = np.array([p * m + j for p in prompt_ids for j in range(m)])
    traj_prompt = np.repeat(np.arange(len(prompt_ids)), m)
    tokens = np.asarray(tokens)[traj][:, :n_steps]
    taken, n_gen = taken_tokens(np.asarray(forced)[traj], tokens, run.cap, eos)
    seed, d, dt = cfg.weight_seed, cfg.d_model, cfg.dtype
    routing = {}

    def get_layer(l):
        lw = M.init_layer(cfg, l, pool=pool)
        say(f"layer {l} ready")
        return lw

    emb = lambda tk: M.init_rows(seed, M.T_EMBED, 0, tk, d, 1, dt)
    last, dec = forced_forward(cfg, np.asarray(prompts)[prompt_ids], traj_prompt, taken[:, :n_steps - 1],
                               get_layer, emb, routing=routing)
    head = M.init_tensor(seed, M.T_LM, 0, cfg.vocab, d, d, dt, pool=pool)
    T = len(traj)
    hid = np.concatenate([last[traj_prompt][:, None, :], dec], axis=1)
    logits = (hid.reshape(T * n_steps, d) @ head.T).reshape(T, n_steps, cfg.vocab)
    del head
    say("logits ready")
    jobs = [(logits[t, s], run.temperature, int(traj[t]), s, run.sample_seed, int(taken[t, s]))
            for t in range(T) for s in range(n_steps)]
    res = pool.map(_score_row, jobs, chunksize=8) if pool is not None else list(map(_score_row, jobs))
    res = np.array(res, dtype=np.float64).reshape(T, n_steps, 5)
    if n_idx >= cfg.vocab:
        idx = np.arange(cfg.vocab)
    else:
        idx = np.sort(np.random.default_rng(idx_seed).choice(cfg.vocab, n_idx, replace=False))
    z = logits / float(run.temperature)
    out = dict(
        prompts=np.array(prompt_ids), traj=traj.astype(np.int32), steps=np.int32(n_steps),
        tokens=tokens.astype(np.int32), taken=taken.astype(np.int32), n_gen=n_gen.astype(np.int32),
        idx=idx.astype(np.int32), logits_at_idx=logits[:, :, idx].astype(np.float32),
        zmax=logits.max(axis=-1), zabs=np.abs(logits).max(axis=-1),
        argmax=logits.argmax(axis=-1).astype(np.int32),
        lse=z.max(axis=-1) + np.log(np.exp(z - z.max(axis=-1, keepdims=True)).sum(axis=-1)),
        sampled=res[..., 0].astype(np.int32), logprob=res[..., 1], entropy=res[..., 2], margin=res[..., 3])
    if cfg.n_experts:
        out["route_ids"] = routing["ids"].astype(np.uint8 if cfg.n_experts <= 256 else np.int32)
        out["route_p"] = routing["p"].astype(np.float32)
        out["route_margin"] = routing["margin"].astype(np.float32)
    return out


def _score_row(args):
    """Sampler outputs of one row: (sample, log-prob, entropy, top-2 margin, 0)."""
    from .sampler import sample_row, top2_margin
    logits, temperature, g, s, seed, force = args
    tok, lp, ent = sample_row(logits, temperature, g, s, seed, force)
    return tok, lp, ent, top2_margin(np.asarray(logits).astype(np.float32), temperature, g, s, seed), 0.0

"""Whole rollout of one batch: prefill, decode steps, scoring, termination,
selection with early stopping, and KV page accounting.

Control flow (paper Alg. 2 applied step by step to a batch decoded together):
* Prefill each prompt; token 0 of every trajectory g = i*m + j is sampled from
  its prompt's last-position logits with counter (g, step 0).
* Each decode step consumes every live trajectory's last token and samples the
  next one (counter (g, s), s = 0-based index of the generated token).
* Termination is exogenous (workload's forced end-of-sequence length d_g): the
  generated token with 1-based count s = d_g <= cap is the end-of-sequence id
  V-1, scored as log p(V-1) under the model; if d_g > cap the trajectory is
  truncated at s = cap (invalid for the long side).  An end-of-sequence id
  sampled earlier is not terminal.
* After every step each unfinished group applies the selection rule
  (oracle.selection.group_decision).  A group that completes aborts its live
  members (tail pruning) and records its step.
* Scores: length = generated count; the log-probability sum is accumulated in
  float32 in step order; mean = fl32(sum / length).

Pages (the KV layout is the HIP path's business; this is the accounting of a
paged pool with page size P_s):
* each prompt holds ceil(Lp / P_s) pages, shared by its m trajectories, freed
  when the last member finishes or is aborted;
* a trajectory that has generated n tokens holds ceil((n-1) / P_s) private
  pages (the newest token's key/value is written when it is consumed); a page
  is taken before the step that writes the first token of a page;
* private pages are freed when the trajectory finishes or is aborted.
The high-water mark is taken after each step's allocations.
"""
from dataclasses import dataclass, field

import numpy as np

from . import model as M
from .sampler import sample_row, top2_margin
from .selection import LIVE, EOS, TRUNC, ABORTED, group_decision


@dataclass
class RolloutResult:
    tokens: dict                 # g -> list of taken tokens
    sampled: dict                # g -> list of sampled tokens (before any force)
    logprobs: dict               # g -> list (float64)
    entropies: dict
    margins: dict                # g -> list of top-2 perturbed-score margins
    route_margins: dict          # g -> list of min MoE routing margin (over layers) per token
    logits: dict                 # g -> list of logit rows (float64) if kept
    status: dict
    length: dict
    sum_lp32: dict
    mean_lp32: dict
    kept: dict                   # prompt -> list of g
    done_step: dict              # prompt -> step
    steps: int
    tokens_decoded: int
    pages_hwm: int
    pages_trace: list            # per step: (n_live_before, pages_after_alloc, pages_after_free)
    live_trace: list


def rollout(cfg, W, prompts, forced, m, k, cap, seed, temperature=1.0, L=1, m_up=None,
            page=16, early_stop=True, prompt_ids=None, keep_logits=False, alloc=None,
            max_steps=None):
    """Run the rollout for prompts ``prompt_ids`` (default all) of the batch.

    prompts: [P, Lp] int; forced: [P*m] raw forced lengths (>= 1).
    Trajectory ids stay global (g = i*m + j) so a subset reproduces the same
    per-trajectory results as the full batch.
    alloc: None (every prompt has m candidates) or the per-prompt redundancy
    plan M'_i <= m of Alg. 1; prompt i then has candidates g = i*m + j,
    j < M'_i, and its group runs shortest-only when M'_i >= m_up, dual-end
    otherwise (Alg. 2).
    max_steps: stop after this many sampling steps even if groups are still
    open (a prefix of the rollout, for checks on long configurations).
    """
    prompts = np.asarray(prompts)
    P, Lp = prompts.shape
    m_up = 2 * k if m_up is None else m_up
    ids = list(range(P)) if prompt_ids is None else list(prompt_ids)
    eos = cfg.vocab - 1
    prompt_pages = -(-Lp // page)

    size = [m] * P if alloc is None else [int(a) for a in alloc]
    trajs = [i * m + j for i in ids for j in range(size[i])]
    st = {g: LIVE for g in trajs}
    gen = {g: 0 for g in trajs}
    toks = {g: [] for g in trajs}
    samp = {g: [] for g in trajs}
    lps = {g: [] for g in trajs}
    ents = {g: [] for g in trajs}
    margins = {g: [] for g in trajs}
    lgs = {g: [] for g in trajs}
    rmar = {g: [] for g in trajs}
    slp = {g: np.float32(0.0) for g in trajs}
    freed = {g: False for g in trajs}
    refcnt = {i: size[i] for i in ids}
    kept, done_step = {}, {}

    # prefill
    caches = {}
    last_logits = {}
    prompt_rmar = {}
    for i in ids:
        mar = []
        lg, cache = M.forward_sequence(cfg, W, prompts[i], margins=mar)
        caches[i] = cache
        last_logits[i] = lg[-1]
        prompt_rmar[i] = float(np.min([m[-1] for m in mar])) if mar else float("inf")
    pages_used = prompt_pages * len(ids)
    hwm = pages_used
    trace, live_trace = [], []

    def emit(g, logits, step_idx):
        s_new = gen[g] + 1
        d = int(forced[g])
        force = eos if (d <= cap and s_new == d) else -1
        tok, lp, ent = sample_row(logits, temperature, g, step_idx, seed, force)
        taken = tok if force < 0 else force
        toks[g].append(taken)
        samp[g].append(tok)
        lps[g].append(lp)
        ents[g].append(ent)
        margins[g].append(top2_margin(np.asarray(logits, np.float64).astype(np.float32),
                                      temperature, g, step_idx, seed))
        if keep_logits:
            lgs[g].append(np.asarray(logits, dtype=np.float64).copy())
        slp[g] = np.float32(slp[g] + np.float32(lp))
        gen[g] = s_new
        if force >= 0:
            st[g] = EOS
        elif s_new >= cap:
            st[g] = TRUNC

    def select_and_free(step):
        nonlocal pages_used
        for i in ids:
            if i in kept:
                continue
            mem = []
            for j in range(size[i]):
                g = i * m + j
                n = gen[g]
                mem.append(dict(g=g, status=st[g], length=n, trunc=(st[g] == TRUNC),
                                mean_lp=float(np.float32(slp[g] / np.float32(max(n, 1))))))
            complete, kp, ab = group_decision(mem, k, L, m_up, early_stop)
            if complete:
                kept[i] = kp
                done_step[i] = step
                for g in ab:
                    st[g] = ABORTED
        for i in ids:
            for j in range(size[i]):
                g = i * m + j
                if st[g] != LIVE and not freed[g]:
                    freed[g] = True
                    pages_used -= -(-(gen[g] - 1) // page) if gen[g] > 1 else 0
                    refcnt[i] -= 1
                    if refcnt[i] == 0:
                        pages_used -= prompt_pages

    # step 1: token 0 from the prompt's logits
    for g in trajs:
        emit(g, last_logits[g // m], 0)
        rmar[g].append(prompt_rmar[g // m])
    trace.append((len(trajs), pages_used, None))
    live_trace.append(len(trajs))
    select_and_free(1)
    trace[-1] = (len(trajs), trace[-1][1], pages_used)

    # per-trajectory caches (contiguous, float64), grouped by prompt
    tcache = {}
    for g in trajs:
        tcache[g] = caches[g // m]
    step = 1
    while len(kept) < len(ids) and (max_steps is None or step < max_steps):
        step += 1
        live = [g for g in trajs if st[g] == LIVE]
        n_before = len(live)
        for g in live:
            if (gen[g] - 1) % page == 0:
                pages_used += 1
        hwm = max(hwm, pages_used)
        alloc_level = pages_used
        if live:
            tok_in = [toks[g][-1] for g in live]
            Lc = [np.stack([tcache[g][l][0] for g in live]) for l in range(cfg.n_layers)]
            Vc = [np.stack([tcache[g][l][1] for g in live]) for l in range(cfg.n_layers)]
            mar = []
            logits, newc = M.decode_batch(cfg, W, tok_in, list(zip(Lc, Vc)), margins=mar)
            rm = np.min(np.stack(mar), axis=0) if mar else np.full(len(live), np.inf)
            for b, g in enumerate(live):
                tcache[g] = [(newc[l][0][b], newc[l][1][b]) for l in range(cfg.n_layers)]
                emit(g, logits[b], gen[g])
                rmar[g].append(float(rm[b]))
        select_and_free(step)
        for g in trajs:
            if st[g] != LIVE and g in tcache:
                del tcache[g]
        trace.append((n_before, alloc_level, pages_used))
        live_trace.append(n_before)

    length = {g: gen[g] for g in trajs}
    mean = {g: np.float32(slp[g] / np.float32(max(gen[g], 1))) for g in trajs}
    return RolloutResult(tokens=toks, sampled=samp, logprobs=lps, entropies=ents, margins=margins,
                         route_margins=rmar,
                         logits=lgs, status=st, length=length, sum_lp32=slp, mean_lp32=mean,
                         kept=kept, done_step=done_step, steps=step,
                         tokens_decoded=sum(length.values()), pages_hwm=hwm,
                         pages_trace=trace, live_trace=live_trace)


def schedule_only(forced, P, m, k, cap, Lp, L=1, m_up=None, page=16, early_stop=True,
                  mean_lp=None, alloc=None):
    """Selection and page accounting without a model.  Termination is exogenous,
    so lengths, completion steps and page counts follow from the forced lengths
    alone; ``mean_lp`` (per trajectory, float32) only breaks length ties.
    ``alloc`` as for rollout(): candidates j >= M'_i of prompt i do not exist
    (status None, length 0)."""
    m_up = 2 * k if m_up is None else m_up
    size = [m] * P if alloc is None else [int(a) for a in alloc]
    n = P * m
    exists = [g % m < size[g // m] for g in range(n)]
    st = [LIVE if exists[g] else None for g in range(n)]
    gen = [1 if exists[g] else 0 for g in range(n)]
    freed = [not exists[g] for g in range(n)]
    refcnt = list(size)
    kept, done_step = {}, {}
    prompt_pages = -(-Lp // page)
    pages = prompt_pages * P
    hwm = pages
    mlp = [0.0] * n if mean_lp is None else [float(x) for x in mean_lp]

    def term(g):
        d = int(forced[g])
        if d <= cap and gen[g] == d:
            st[g] = EOS
        elif gen[g] >= cap:
            st[g] = TRUNC

    def sel(step):
        nonlocal pages
        for i in range(P):
            if i in kept:
                continue
            mem = [dict(g=g, status=st[g], length=gen[g], trunc=st[g] == TRUNC, mean_lp=mlp[g])
                   for g in range(i * m, i * m + size[i])]
            c, kp, ab = group_decision(mem, k, L, m_up, early_stop)
            if c:
                kept[i] = kp
                done_step[i] = step
                for g in ab:
                    st[g] = ABORTED
        for g in range(n):
            if exists[g] and st[g] != LIVE and not freed[g]:
                freed[g] = True
                pages -= -(-(gen[g] - 1) // page)
                refcnt[g // m] -= 1
                if refcnt[g // m] == 0:
                    pages -= prompt_pages

    for g in range(n):
        if exists[g]:
            term(g)
    sel(1)
    step = 1
    decoded = sum(size)
    while len(kept) < P:
        step += 1
        live = [g for g in range(n) if st[g] == LIVE]
        for g in live:
            if (gen[g] - 1) % page == 0:
                pages += 1
        hwm = max(hwm, pages)
        for g in live:
            gen[g] += 1
            decoded += 1
            term(g)
        sel(step)
    return dict(kept=kept, done_step=done_step, steps=step, tokens_decoded=decoded,
                pages_hwm=hwm, pages_end=pages, length=list(gen), status=list(st))

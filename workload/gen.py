"""Seeded generators.  Draw order is fixed so every run reproduces the same data."""
import numpy as np

from .configs import ModelCfg, RunCfg, SWEEP


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest even); return uint16 bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (b >> 16) & 1
    r = ((b + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        r = np.where(nan, np.uint16(0x7FC0), r)
    return r


def f32_from_bf16_bits(h: np.ndarray) -> np.ndarray:
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def rollout_inputs(model: ModelCfg, run: RunCfg):
    """Prompt tokens [P, Lp] (int32) and raw forced end-of-sequence draws [P*m] (int32, >= 1).

    Lengths are lognormal(ln median, sigma); with ``len_tail`` a Bernoulli(0.05)
    replaces a draw by U(5, 10) x median.  Trajectory g = i*m + j belongs to prompt i.
    """
    rng = np.random.default_rng(run.workload_seed)
    P, m = run.n_prompts, run.m
    prompts = rng.integers(0, model.vocab, size=(P, run.prompt_len), dtype=np.int64)
    z = rng.standard_normal(P * m)
    raw = run.len_median * np.exp(run.len_sigma * z)
    if run.len_tail:
        tu = rng.random(P * m)
        tf = rng.uniform(5.0, 10.0, P * m)
        raw = np.where(tu < 0.05, run.len_median * tf, raw)
    d = np.maximum(1, np.rint(raw)).astype(np.int64)
    d = np.minimum(d, 1 << 30)
    return prompts.astype(np.int32), d.astype(np.int32)


def heterogeneous_forced_lengths(run: RunCfg, seed: int, sigmas=(0.3, 1.2)):
    """Raw forced end-of-sequence draws [P*m] (int32, >= 1) whose spread
    belongs to the prompt, as with prompts of unequal difficulty: prompt i
    draws lognormal(ln median, sigmas[i % len(sigmas)]) lengths, and only the
    prompts of the largest sigma have the Bernoulli(0.05) tail at U(5, 10) x
    median (with ``len_tail``).  Used to exercise the adaptive allocation,
    which needs a spread that persists per prompt."""
    rng = np.random.default_rng(seed)
    P, m = run.n_prompts, run.m
    sig = np.repeat(np.array([sigmas[i % len(sigmas)] for i in range(P)], dtype=np.float64), m)
    z = rng.standard_normal(P * m)
    raw = run.len_median * np.exp(sig * z)
    if run.len_tail:
        tu = rng.random(P * m)
        tf = rng.uniform(5.0, 10.0, P * m)
        raw = np.where((tu < 0.05) & (sig == max(sigmas)), run.len_median * tf, raw)
    d = np.maximum(1, np.rint(raw)).astype(np.int64)
    return np.minimum(d, 1 << 30).astype(np.int32)


def sweep_attention_inputs(rows=None, seed=None):
    """Context lengths [rows] (int32) and a page permutation seed for the attention sweep."""
    s = SWEEP
    rows = s["attn_rows"] if rows is None else rows
    seed = s["seed"] if seed is None else seed
    rng = np.random.default_rng([seed, 0])
    ctx = np.rint(s["attn_ctx_median"] * np.exp(s["attn_ctx_sigma"] * rng.standard_normal(rows)))
    ctx = np.clip(ctx, s["attn_ctx_min"], s["attn_ctx_max"]).astype(np.int32)
    return ctx, rng


def sweep_page_table(ctx: np.ndarray, page: int, rng, spare: int = 0):
    """Page table [rows, max_pages] (int32, -1 padded) drawing page ids from a shuffled pool."""
    npg = (ctx.astype(np.int64) + page - 1) // page
    total = int(npg.sum()) + spare
    perm = rng.permutation(total).astype(np.int32)
    maxp = int(npg.max()) if len(npg) else 1
    pt = np.full((len(ctx), maxp), -1, dtype=np.int32)
    off = 0
    for r, n in enumerate(npg):
        pt[r, :n] = perm[off:off + n]
        off += n
    return pt, total


def shared_prefix_page_table(group_sizes, m, prefix_pages, ctx, page, rng, spare=0):
    """Rows of prompt groups that share their first ``prefix_pages`` pages.

    Group i has ``group_sizes[i]`` members (a sorted random subset of the m
    trajectory slots, traj = i*m + j); every member's page-table row starts
    with the group's prefix pages, then holds private pages for the rest of
    ``ctx`` keys.  Page ids come from a shuffled pool.  Returns (row_traj
    [n_rows] int32, page table [n_groups*m, max_pages] int32 (-1 for unused),
    pool size)."""
    npg = (int(ctx) + page - 1) // page
    priv = npg - prefix_pages
    n_rows = int(sum(group_sizes))
    total = len(group_sizes) * prefix_pages + n_rows * priv + spare
    perm = rng.permutation(total).astype(np.int32)
    pt = np.full((len(group_sizes) * m, npg), -1, dtype=np.int32)
    rows = []
    off = 0
    for i, n in enumerate(group_sizes):
        shared = perm[off:off + prefix_pages]
        off += prefix_pages
        for j in np.sort(rng.choice(m, size=n, replace=False)):
            g = i * m + int(j)
            pt[g, :prefix_pages] = shared
            pt[g, prefix_pages:] = perm[off:off + priv]
            off += priv
            rows.append(g)
    return np.asarray(rows, dtype=np.int32), pt, total


def sweep_sampler_logits(rows=None, vocab=None, seed=None) -> np.ndarray:
    """bf16 logits ~ N(0, std) as uint16 bit patterns [rows, vocab]."""
    s = SWEEP
    rows = s["samp_rows"] if rows is None else rows
    vocab = s["samp_vocab"] if vocab is None else vocab
    seed = s["seed"] if seed is None else seed
    rng = np.random.default_rng([seed, 1])
    out = np.empty((rows, vocab), dtype=np.uint16)
    for r in range(rows):
        out[r] = bf16_bits_from_f32(rng.normal(0.0, s["samp_std"], vocab).astype(np.float32))
    return out


def sweep_selection_inputs(n=None, seed=None, cap=None, median=None):
    """Raw lengths (int32 >= 1) and mean log-probs on a 2^-10 grid (float32, exact ties)."""
    s = SWEEP
    n = s["sel_traj"] if n is None else n
    seed = s["seed"] if seed is None else seed
    median = s["sel_len_median"] if median is None else median
    rng = np.random.default_rng([seed, 2])
    raw = np.maximum(1, np.rint(median * np.exp(rng.standard_normal(n)))).astype(np.int32)
    mlp = -(np.floor(rng.random(n) * 3 * 1024) / 1024).astype(np.float32)
    return raw, mlp


def synthetic_rewards(n, seed, p_correct=0.5):
    """Verifiable-reward stand-in: float32 {0, 1} per trajectory, Bernoulli(p_correct)."""
    rng = np.random.default_rng([seed, 7])
    return (rng.random(n) < p_correct).astype(np.float32)


def teacher_forcing_tokens(model: ModelCfg, run: RunCfg, n_steps: int) -> np.ndarray:
    """Token table [P*m, n_steps] (int32) for teacher-forced parity runs: row g
    holds the tokens trajectory g takes at generated indices 0 .. n_steps-1,
    uniform over [0, vocab-1) (the end-of-sequence id vocab-1 only comes from
    the forced lengths).  Drawn independently of both sides' samplers."""
    rng = np.random.default_rng([run.workload_seed, 5])
    return rng.integers(0, model.vocab - 1, size=(run.n_prompts * run.m, n_steps)).astype(np.int32)


def sweep_selection_pages(length, page=16, seed=None):
    """KV page lists of the selection sweep's trajectories, CSR: trajectory g
    holds ceil(length[g] / page) ids, pages[off[g] : off[g+1]], drawn from a
    shuffled pool.  Returns (off [n+1] int32, pages [total] int32)."""
    s = SWEEP
    seed = s["seed"] if seed is None else seed
    rng = np.random.default_rng([seed, 3])
    npg = (np.asarray(length, dtype=np.int64) + page - 1) // page
    off = np.concatenate([[0], np.cumsum(npg)]).astype(np.int32)
    return off, rng.permutation(int(npg.sum())).astype(np.int32)

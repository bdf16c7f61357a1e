"""Kernel parity on the GPU through the C ABI: Gumbel map (bit-exact over all
2^23 inputs), fused sampler (tokens bit-exact, log-prob/entropy within
tolerance), paged decode attention, selection (bit-exact kept sets).  Every
expected value comes from oracle/ on the same seeded inputs."""
import math
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle.fp32math import gumbel_f32
from oracle.sampler import sample_row
from oracle.selection import group_decision, reclaimed_pages, LIVE, EOS, TRUNC, ABORTED
from oracle import sweep as OS
from workload import sweep_attention_inputs, sweep_sampler_logits, sweep_selection_inputs
from workload.gen import (sweep_page_table, shared_prefix_page_table, f32_from_bf16_bits,
                          sweep_selection_pages)
from workload.configs import SWEEP

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _b():
    from paper_2605_30859_amd import binding
    binding.load_library()
    return binding


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def test_gumbel_map_bit_exact_all_u():
    B = _b()
    say("gumbel map: 2^23 inputs")
    k = np.arange(1 << 23, dtype=np.uint64) * 2 + 1
    u = (k.astype(np.float32) * np.float32(2.0 ** -24)).astype(np.float32)
    ref = gumbel_f32(u)
    ud = torch.from_numpy(u).to(DEV)
    gd = torch.empty_like(ud)
    B.darts_debug_gumbel(ud, gd)
    torch.cuda.synchronize()
    got = gd.cpu().numpy()
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_gumbel_fast_map_within_filter_bound_all_u():
    """The sampler pre-selects candidates with a fast Gumbel map and only the
    exact map decides; that is sound if the fast map stays within the bound
    the filter assumes on every one of the 2^23 possible u."""
    B = _b()
    say("fast gumbel map: 2^23 inputs")
    k = np.arange(1 << 23, dtype=np.uint64) * 2 + 1
    u = (k.astype(np.float32) * np.float32(2.0 ** -24)).astype(np.float32)
    ud = torch.from_numpy(u).to(DEV)
    exact, fast = torch.empty_like(ud), torch.empty_like(ud)
    B.darts_debug_gumbel(ud, exact)
    B.darts_debug_gumbel_fast(ud, fast)
    torch.cuda.synchronize()
    err = (fast.double() - exact.double()).abs().max().item()
    bound = B.darts_sampler_gumbel_bound()
    say(f"fast gumbel map: max |fast - exact| = {err:.3e}, filter bound {bound:.3e}")
    assert np.array_equal(exact.cpu().numpy().view(np.uint32), gumbel_f32(u).view(np.uint32))
    assert err <= bound


def test_sampler_filter_near_ties():
    """Logits built from the oracle's own Gumbel noise so that several
    perturbed scores tie exactly or within a few ulp: in one thread's
    elements (4 consecutive ids, ids 1024 apart), across threads, and a
    unique winner one ulp above a same-thread runner-up.  These take the
    sampler's exact re-scan; the token must still be the oracle's
    first-maximal index."""
    from oracle.sampler import gumbel_noise
    B = _b()
    rows, vocab, seed = 16, 4096, 424242
    rng = np.random.default_rng(3)
    l32 = (rng.normal(0, 1, (rows, vocab)) - 30.0).astype(np.float32)
    traj = np.arange(rows, dtype=np.int32) * 5 + 1
    step = np.arange(rows, dtype=np.int32) % 3
    C = np.float32(5.0)
    for r in range(rows):
        g = gumbel_noise(vocab, int(traj[r]), int(step[r]), seed)
        kind = r % 4
        if kind == 0:      # one thread: ids 4j..4j+3 and 4(j+256)+1
            j = int(rng.integers(0, 256))
            picks = [4 * j, 4 * j + 1, 4 * j + 2, 4 * j + 3, 4 * (j + 256) + 1]
        elif kind == 1:    # several threads
            picks = [int(x) for x in rng.choice(vocab, 6, replace=False)]
        else:              # a runner-up within one ulp, same thread (2) or not (3)
            j = int(rng.integers(0, 256))
            picks = [4 * j + 2, 4 * (j + 512)] if kind == 2 else [4 * j + 2, 4 * ((j + 7) % 256) + 3]
        for i in picks:
            l32[r, i] = np.float32(C - g[i])
        if kind >= 2:
            l32[r, picks[1]] = np.nextafter(l32[r, picks[1]], np.float32(np.inf))
    logits = torch.from_numpy(l32).to(DEV)
    td, sd = torch.from_numpy(traj).to(DEV), torch.from_numpy(step).to(DEV)
    tok = torch.empty(rows, dtype=torch.int32, device=DEV)
    lp = torch.empty(rows, dtype=torch.float32, device=DEV)
    ent = torch.empty(rows, dtype=torch.float32, device=DEV)
    B.darts_sample(logits, B.DARTS_F32, seed, td, sd, 1.0, None, tok, lp, ent)
    torch.cuda.synchronize()
    tok, lp, ent = tok.cpu().numpy(), lp.cpu().numpy(), ent.cpu().numpy()
    for r in range(rows):
        stok, slp, sent = sample_row(l32[r], 1.0, int(traj[r]), int(step[r]), seed)
        assert tok[r] == stok, (r, tok[r], stok)
        assert abs(lp[r] - slp) < 1e-4 and abs(ent[r] - sent) < 1e-4


def test_sampler_edge_rows():
    """Degenerate rows, each against the oracle: the smallest vocabulary
    (V = 4), one logit 40 above the rest (entropy ~ 0, log-prob ~ 0), masked
    rows with only 3 finite logits (the token is one of them, scores are
    those of the finite sub-vocabulary), a row whose first 1024 logits are
    masked (whole threads see only -inf), and equal logits."""
    B = _b()
    seed = 31337
    cases = []
    rng = np.random.default_rng(9)
    cases.append(rng.normal(0, 2, 4).astype(np.float32))
    z = rng.normal(0, 1, 2048).astype(np.float32)
    z[777] = 40.0
    cases.append(z)
    z = np.full(4096, -np.inf, dtype=np.float32)
    z[[5, 2049, 4095]] = [0.5, -1.0, 0.25]
    cases.append(z)
    z = rng.normal(0, 1, 4096).astype(np.float32)
    z[:1024] = -np.inf
    cases.append(z)
    cases.append(np.zeros(4096, dtype=np.float32))
    for ci, z in enumerate(cases):
        V = len(z)
        traj = torch.tensor([ci * 3 + 1], dtype=torch.int32, device=DEV)
        step = torch.tensor([ci], dtype=torch.int32, device=DEV)
        tok = torch.empty(1, dtype=torch.int32, device=DEV)
        lp = torch.empty(1, dtype=torch.float32, device=DEV)
        ent = torch.empty(1, dtype=torch.float32, device=DEV)
        B.darts_sample(torch.from_numpy(z).to(DEV).view(1, V), B.DARTS_F32, seed, traj, step, 1.0, None,
                       tok, lp, ent)
        torch.cuda.synchronize()
        stok, slp, sent = sample_row(z, 1.0, ci * 3 + 1, ci, seed)
        assert int(tok.item()) == stok, (ci, int(tok.item()), stok)
        assert np.isfinite(lp.item()) and np.isfinite(ent.item()), ci
        assert abs(lp.item() - slp) < 1e-5 and abs(ent.item() - sent) < 1e-5, (ci, lp.item(), slp, ent.item(), sent)
        if ci == 1:
            assert stok == 777 and ent.item() < 1e-6
        if ci == 2:
            assert stok in (5, 2049, 4095)


def test_sampler_rows_without_finite_score():
    """Rows whose every logit is -inf or NaN have no Gumbel-max winner: the
    token is 0 (the lowest index, as the oracle's first-maximum argmax gives
    for equal scores), a teacher-forced token is still taken, and log-prob
    and entropy are NaN on both sides.  Ordinary rows in the same launch are
    unaffected."""
    B = _b()
    V, seed = 4096, 77
    rng = np.random.default_rng(21)
    z = rng.normal(0, 1, (5, V)).astype(np.float32)
    z[1] = -np.inf
    z[2] = np.nan
    z[3] = -np.inf
    force = np.array([-1, -1, -1, 17, -1], dtype=np.int32)
    traj = torch.arange(5, dtype=torch.int32, device=DEV) + 40
    step = torch.full((5,), 3, dtype=torch.int32, device=DEV)
    tok = torch.empty(5, dtype=torch.int32, device=DEV)
    lp = torch.empty(5, dtype=torch.float32, device=DEV)
    ent = torch.empty(5, dtype=torch.float32, device=DEV)
    B.darts_sample(torch.from_numpy(z).to(DEV), B.DARTS_F32, seed, traj, step, 1.0,
                   torch.from_numpy(force).to(DEV), tok, lp, ent)
    torch.cuda.synchronize()
    tok, lp, ent = tok.cpu().numpy(), lp.cpu().numpy(), ent.cpu().numpy()
    for r in range(5):
        stok, slp, sent = sample_row(z[r], 1.0, 40 + r, 3, seed, int(force[r]))
        taken = stok if force[r] < 0 else int(force[r])
        assert tok[r] == taken, (r, tok[r], taken)
        if r in (1, 2, 3):
            assert stok == 0 and np.isnan(slp) and np.isnan(sent)
            assert np.isnan(lp[r]) and np.isnan(ent[r]), (r, lp[r], ent[r])
        else:
            assert abs(lp[r] - slp) < 1e-5 and abs(ent[r] - sent) < 1e-5, r


def _bf16_tensor(bits):
    return torch.from_numpy(bits.view(np.int16)).to(DEV).view(torch.bfloat16)


@pytest.mark.parametrize("dtype,rows,vocab,temp", [("bf16", 64, 4096, 1.0), ("f32", 48, 512, 1.0),
                                                  ("f32", 33, 1000, 0.7), ("bf16", 7, 32000, 1.3)])
def test_sampler_small(dtype, rows, vocab, temp):
    B = _b()
    say(f"sampler {dtype} rows={rows} V={vocab} T={temp}")
    bits = sweep_sampler_logits(rows=rows, vocab=vocab, seed=5)
    l32 = f32_from_bf16_bits(bits)
    if dtype == "bf16":
        logits = _bf16_tensor(bits)
        dt = B.DARTS_BF16
    else:
        rng = np.random.default_rng(11)
        l32 = (l32 + rng.normal(0, 1e-3, l32.shape)).astype(np.float32)   # not bf16-exact
        logits = torch.from_numpy(l32).to(DEV)
        dt = B.DARTS_F32
    traj = torch.arange(rows, dtype=torch.int32, device=DEV) * 7 + 3
    step = torch.arange(rows, dtype=torch.int32, device=DEV) % 5
    force = torch.full((rows,), -1, dtype=torch.int32, device=DEV)
    force[::3] = torch.arange(0, rows, 3, dtype=torch.int32, device=DEV) % vocab
    tok = torch.empty(rows, dtype=torch.int32, device=DEV)
    lp = torch.empty(rows, dtype=torch.float32, device=DEV)
    ent = torch.empty(rows, dtype=torch.float32, device=DEV)
    seed = 1234567
    B.darts_sample(logits, dt, seed, traj, step, temp, force, tok, lp, ent)
    torch.cuda.synchronize()
    tok, lp, ent = tok.cpu().numpy(), lp.cpu().numpy(), ent.cpu().numpy()
    tr, sp, fo = traj.cpu().numpy(), step.cpu().numpy(), force.cpu().numpy()
    for r in range(rows):
        stok, slp, sent = sample_row(l32[r], temp, int(tr[r]), int(sp[r]), seed, int(fo[r]))
        taken = stok if fo[r] < 0 else int(fo[r])
        assert tok[r] == taken, (r, tok[r], taken)
        assert abs(lp[r] - slp) < 1e-4, (r, lp[r], slp)
        assert abs(ent[r] - sent) < 1e-4, (r, ent[r], sent)


def test_sampler_full_sweep_size():
    """1024 x 151936 bf16 logits ~ N(0, 3) (the sweep's shape); tokens
    bit-exact on every 8th row and the last, log-prob and entropy within
    1e-3."""
    B = _b()
    rows, vocab = SWEEP["samp_rows"], SWEEP["samp_vocab"]
    say(f"sampler sweep {rows}x{vocab}")
    bits = sweep_sampler_logits()
    logits = _bf16_tensor(bits)
    traj = torch.arange(rows, dtype=torch.int32, device=DEV)
    step = torch.zeros(rows, dtype=torch.int32, device=DEV)
    tok = torch.empty(rows, dtype=torch.int32, device=DEV)
    lp = torch.empty(rows, dtype=torch.float32, device=DEV)
    ent = torch.empty(rows, dtype=torch.float32, device=DEV)
    seed = SWEEP["seed"]
    B.darts_sample(logits, B.DARTS_BF16, seed, traj, step, 1.0, None, tok, lp, ent)
    torch.cuda.synchronize()
    tok, lp, ent = tok.cpu().numpy(), lp.cpu().numpy(), ent.cpu().numpy()
    l32 = None
    for r in list(range(0, rows, 8)) + [rows - 1]:
        row = f32_from_bf16_bits(bits[r])
        stok, slp, sent = sample_row(row, 1.0, r, 0, seed)
        assert tok[r] == stok
        assert abs(lp[r] - slp) < 1e-3 and abs(ent[r] - sent) < 1e-3
    # properties at any size: entropy within [0, ln V], log-prob <= 0
    assert (ent >= 0).all() and (ent <= math.log(vocab) + 1e-3).all()
    assert (lp <= 1e-6).all()


def _attn_case(rows, hq, hkv, hd, ctx, dtype, seed, spare=3, equal=False):
    B = _b()
    rng = np.random.default_rng(seed)
    pt, n_pages = sweep_page_table(ctx, 16, rng, spare=spare)
    max_ctx = int(ctx.max())
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dt = B.DARTS_BF16 if dtype == "bf16" else B.DARTS_F32
    q = torch.empty(rows * hq * hd, dtype=tdt, device=DEV)
    kp = torch.empty(n_pages * hkv * 16 * hd, dtype=tdt, device=DEV)
    vp = torch.empty_like(kp)
    B.darts_fill_uniform(q, OS.T_Q, seed, dt)
    B.darts_fill_kv_pool(kp, vp, n_pages, hkv, hd, seed, dt)
    ptd = torch.from_numpy(pt).to(DEV)
    ctxd = torch.from_numpy(ctx.astype(np.int32)).to(DEV)
    out = torch.zeros(rows * hq * hd, dtype=tdt, device=DEV)
    ws = torch.empty(B.darts_attn_workspace_bytes(rows, hq, hkv, hd, max_ctx), dtype=torch.uint8,
                     device=DEV)
    B.darts_attn_decode(q, kp, vp, n_pages, ptd, None if equal else ctxd, hq, hkv, hd, max_ctx, dt,
                        out, ws, n_rows=rows)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().reshape(rows, hq, hd), pt


@pytest.mark.parametrize("dtype,hq,hkv,hd", [("bf16", 32, 8, 128), ("bf16", 16, 4, 64),
                                            ("bf16", 8, 8, 128), ("bf16", 32, 4, 128),
                                            ("f32", 4, 4, 32), ("f32", 8, 2, 64)])
def test_attention_small_ragged(dtype, hq, hkv, hd):
    """Ragged contexts (1 .. several chunks, partial last pages) in a shuffled pool."""
    say(f"attention {dtype} hq={hq} hkv={hkv} hd={hd}")
    ctx = np.array([1, 15, 16, 17, 31, 33, 100, 257, 513, 1024, 1500, 2049, 3000, 40, 5, 700],
                   dtype=np.int64)
    rows = len(ctx)
    seed = 77
    got, pt = _attn_case(rows, hq, hkv, hd, ctx, dtype, seed)
    tol = 2e-2 if dtype == "bf16" else 1e-5
    for r in range(rows):
        ref = OS.attention_row(r, int(ctx[r]), pt[r], seed, hq, hkv, hd)
        err = np.max(np.abs(got[r] - ref))
        assert err <= tol * max(1.0, np.max(np.abs(ref))), (r, ctx[r], err)


@pytest.mark.parametrize("rows,hq,hkv,hd,ctx", [
    (1, 32, 8, 128, 700),
    (63, 32, 8, 128, 257),      # one row below the double-buffered form; odd page count
    (64, 32, 8, 128, 257),      # the first double-buffered batch size
    (64, 32, 8, 128, 17),       # one page pair, one key in its second page
    (100, 32, 8, 128, 16),      # one page, no second page in the pair
    (130, 32, 8, 128, 4111),    # rows split into chunks, combine
    (512, 32, 8, 128, 1200),    # the rollout's first-step batch
    (96, 16, 4, 64, 1500),
    (80, 8, 8, 128, 33),        # G = 1
    (72, 8, 2, 32, 600),
    (256, 32, 4, 128, 1500),    # the MoE shape's heads (G = 8), double-buffered
    (20, 32, 4, 128, 3001),     # G = 8, few rows: context chunks and combine
])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_attention_equal_contexts(rows, hq, hkv, hd, ctx, dtype):
    """The equal-context form a decode step takes (no per-row contexts; in
    bf16 the work is mapped arithmetically, with double-buffered page pairs
    from 64 rows) against the oracle, on every row or a sample of them."""
    say(f"attention equal contexts {dtype} rows={rows} hq={hq} hkv={hkv} hd={hd} ctx={ctx}")
    seed = 123
    c = np.full(rows, ctx, dtype=np.int64)
    got, pt = _attn_case(rows, hq, hkv, hd, c, dtype, seed, equal=True)
    tol = 2e-2 if dtype == "bf16" else 1e-5
    sample = range(rows) if rows <= 64 else sorted({0, 1, rows // 2, rows - 1, *range(0, rows, 37)})
    for r in sample:
        ref = OS.attention_row(r, ctx, pt[r], seed, hq, hkv, hd)
        err = np.max(np.abs(got[r] - ref))
        assert err <= tol * max(1.0, np.max(np.abs(ref))), (r, err)
    assert np.isfinite(got).all()


def test_attention_full_sweep_sampled_rows():
    """The sweep's shape: 1024 trajectories, 32/8 heads, hd 128, lognormal
    contexts in [16, 32768] over a shuffled pool; sampled rows vs the oracle."""
    say("attention sweep full size")
    ctx, rng = sweep_attention_inputs()
    seed = SWEEP["seed"]
    got, pt = _attn_case(len(ctx), 32, 8, 128, ctx.astype(np.int64), "bf16", seed)
    order = np.argsort(ctx)
    sample = list(order[:3]) + list(order[-3:]) + list(range(0, len(ctx), 151))
    for r in sample:
        ref = OS.attention_row(int(r), int(ctx[r]), pt[r], seed, 32, 8, 128)
        err = np.max(np.abs(got[r] - ref))
        assert err <= 2e-2 * max(1.0, np.max(np.abs(ref))), (r, ctx[r], err)
    assert np.isfinite(got).all()


@pytest.mark.parametrize("hq,hkv,hd,m,prefix_pages,extra,groups", [
    (32, 8, 128, 16, 32, 600, (16, 5, 1, 16, 9)),     # Qwen3-8B heads; suffix split in chunks
    (32, 4, 128, 16, 13, 1, (3, 16)),                # G = 8; prefix chunks 8 + 5; one suffix key
    (16, 4, 64, 16, 2, 37, (16, 16, 7)),             # dense-small heads
    (8, 8, 128, 8, 3, 20, (8, 2)),                   # G = 1
    (32, 8, 128, 16, 32, 100, (16,) * 32),           # 512 rows (the rollout's first steps)
    (32, 8, 128, 16, 32, 7687, (8,)),                # few rows, long suffix: 61 chunks per row
])
def test_attention_shared_prefix(hq, hkv, hd, m, prefix_pages, extra, groups):
    """Rows of prompt groups sharing their prompt pages: the shared-prefix
    path against the oracle (sampled rows for the 512-row case) and against
    the per-row path on the same inputs."""
    B = _b()
    seed = 91
    ctx = prefix_pages * 16 + extra
    say(f"shared-prefix attention hq={hq} hkv={hkv} hd={hd} m={m} pp={prefix_pages} ctx={ctx} groups={groups}")
    rng = np.random.default_rng(seed)
    row_traj, pt, n_pages = shared_prefix_page_table(groups, m, prefix_pages, ctx, 16, rng, spare=5)
    rows = len(row_traj)
    q = torch.empty(rows * hq * hd, dtype=torch.bfloat16, device=DEV)
    kp = torch.empty(n_pages * hkv * 16 * hd, dtype=torch.bfloat16, device=DEV)
    vp = torch.empty_like(kp)
    B.darts_fill_uniform(q, OS.T_Q, seed, B.DARTS_BF16)
    B.darts_fill_kv_pool(kp, vp, n_pages, hkv, hd, seed, B.DARTS_BF16)
    ptd = torch.from_numpy(pt).to(DEV)
    rtd = torch.from_numpy(row_traj).to(DEV)
    out = torch.zeros(rows * hq * hd, dtype=torch.bfloat16, device=DEV)
    ws = torch.empty(B.darts_attn_shared_workspace_bytes(rows, hq, hkv, hd, ctx, prefix_pages),
                     dtype=torch.uint8, device=DEV)
    B.darts_attn_decode_shared(q, kp, vp, n_pages, ptd, rtd, m, prefix_pages, ctx, hq, hkv, hd,
                               B.DARTS_BF16, out, ws)
    # the per-row path on the same rows (page-table rows gathered per row)
    pt_rows = torch.from_numpy(np.ascontiguousarray(pt[row_traj])).to(DEV)
    ctxd = torch.full((rows,), ctx, dtype=torch.int32, device=DEV)
    out2 = torch.zeros_like(out)
    ws2 = torch.empty(B.darts_attn_workspace_bytes(rows, hq, hkv, hd, ctx), dtype=torch.uint8, device=DEV)
    B.darts_attn_decode(q, kp, vp, n_pages, pt_rows, ctxd, hq, hkv, hd, ctx, B.DARTS_BF16, out2, ws2)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().reshape(rows, hq, hd)
    got2 = out2.float().cpu().numpy().reshape(rows, hq, hd)
    assert np.isfinite(got).all()
    assert np.max(np.abs(got - got2)) <= 2e-2 * max(1.0, np.max(np.abs(got2)))
    if ctx > 4096:
        sample = [0, rows - 1]
    else:
        sample = range(rows) if rows <= 64 else list(range(0, rows, 37)) + [rows - 1]
    for r in sample:
        ref = OS.attention_row(r, ctx, pt[row_traj[r]], seed, hq, hkv, hd)
        err = np.max(np.abs(got[r] - ref))
        assert err <= 2e-2 * max(1.0, np.max(np.abs(ref))), (r, err)


def test_attention_shared_prefix_errors():
    B = _b()
    q = torch.zeros(4 * 32 * 128, dtype=torch.bfloat16, device=DEV)
    kp = torch.zeros(64 * 8 * 16 * 128, dtype=torch.bfloat16, device=DEV)
    pt = torch.zeros((16, 8), dtype=torch.int32, device=DEV)
    rt = torch.arange(4, dtype=torch.int32, device=DEV)
    ws = torch.empty(1 << 20, dtype=torch.uint8, device=DEV)
    with pytest.raises(B.DartsError):   # context not beyond the prefix
        B.darts_attn_decode_shared(q, kp, kp, 64, pt, rt, 4, 2, 32, 32, 8, 128, B.DARTS_BF16, q, ws)
    with pytest.raises(B.DartsError):   # fp32 is not supported on this path
        B.darts_attn_decode_shared(q, kp, kp, 64, pt, rt, 4, 2, 40, 32, 8, 128, B.DARTS_F32, q, ws)
    with pytest.raises(B.DartsError):   # workspace too small
        B.darts_attn_decode_shared(q, kp, kp, 64, pt, rt, 4, 2, 40, 32, 8, 128, B.DARTS_BF16, q, ws[:64])


def _oracle_select(status, length, mlp, m, k, L, m_up, early_stop):
    n = len(status)
    kept = {}
    new_status = status.copy()
    for grp in range(n // m):
        mem = []
        for j in range(m):
            g = grp * m + j
            mem.append(dict(g=g, status=int(status[g]), length=int(length[g]),
                            trunc=int(status[g]) == TRUNC, mean_lp=float(mlp[g])))
        c, kp, ab = group_decision(mem, k, L, m_up, early_stop)
        if c:
            kept[grp] = kp
            for g in ab:
                new_status[g] = ABORTED
    return kept, new_status


@pytest.mark.parametrize("mode", ["short_final", "short_mid", "dual_final", "dual_mid", "no_abort_mid"])
def test_selection_sweep(mode):
    """65536 trajectories in groups of m=16, k=8 (L=1), lengths lognormal,
    mean log-probs on a 2^-10 grid (exact ties): kept sets and statuses
    bit-exact, and the page ids the completed groups free (ceil(len/16) per
    trajectory from a shuffled pool) bit-exact in order and count."""
    _selection_case(mode, SWEEP["sel_m"], SWEEP["sel_k"], 1, None)


@pytest.mark.parametrize("mode", ["short_mid", "dual_mid", "dual_final"])
def test_selection_full_wavefront_groups(mode):
    """Groups of the largest size, m = 64 (one full wavefront per group),
    k = 32, L = 3; 16384 trajectories: the same bit-exact checks."""
    _selection_case(mode, 64, 32, 3, 16384)


def _selection_case(mode, m, k, L, n_traj):
    B = _b()
    say(f"selection {mode}, m {m}, k {k}, L {L}")
    raw, mlp = sweep_selection_inputs(n=n_traj)
    cap = SWEEP["sel_cap"]
    m_up = m if mode.startswith("short") or mode.startswith("no_abort") else m + 1
    early = 0 if mode.startswith("no_abort") else 1
    length = np.minimum(raw, cap).astype(np.int32)
    trunc = raw > cap
    if mode.endswith("final"):
        s = cap
    elif m_up <= m and early:
        s = int(np.median(length))
    else:
        # modes that wait for every member: a step at which about half the
        # groups are done (a quarter when half of the groups reach the cap)
        gmax = length.reshape(-1, m).max(axis=1)
        s = int(np.median(gmax))
        if s >= cap:
            s = int(np.percentile(gmax, 25))
    status = np.where(length <= s, np.where(trunc, TRUNC, EOS), LIVE).astype(np.uint8)
    cur_len = np.minimum(length, s).astype(np.int32)
    kept_ref, st_ref = _oracle_select(status, cur_len, mlp, m, k, L, m_up, early)
    n = len(status)
    st_d = torch.from_numpy(status).to(DEV)
    len_d = torch.from_numpy(cur_len).to(DEV)
    mlp_d = torch.from_numpy(mlp).to(DEV)
    kept_d = torch.full((n // m, k), -1, dtype=torch.int32, device=DEV)
    comp_d = torch.zeros(n // m, dtype=torch.uint8, device=DEV)
    # page lists: ceil(len / 16) ids per trajectory (its length at this step)
    off, pages = sweep_selection_pages(cur_len)
    off_d, pages_d = torch.from_numpy(off).to(DEV), torch.from_numpy(pages).to(DEV)
    free_d = torch.full((len(pages),), -1, dtype=torch.int32, device=DEV)
    nfree_d = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    work_d = torch.empty(n // m + 1, dtype=torch.int32, device=DEV)
    B.darts_select_groups(st_d, len_d, mlp_d, m, k, L, m_up, early, kept_d, comp_d, off_d, pages_d,
                          free_d, nfree_d, work_d)
    torch.cuda.synchronize()
    kept, comp, st = kept_d.cpu().numpy(), comp_d.cpu().numpy(), st_d.cpu().numpy()
    assert np.array_equal(st, st_ref)
    for grp in range(n // m):
        if grp in kept_ref:
            assert comp[grp] == 1
            assert list(kept[grp]) == kept_ref[grp], grp
        else:
            assert comp[grp] == 0 and (kept[grp] == -1).all()
    assert len(kept_ref) > 0
    # reclaimed pages: bit-exact list and count (the oracle's group / member / list order)
    lists = [pages[off[g]:off[g + 1]] for g in range(n)]
    want = np.array(reclaimed_pages(lists, set(kept_ref), m), dtype=np.int32)
    nf = int(nfree_d.item())
    free = free_d.cpu().numpy()
    say(f"selection {mode} m {m}: {len(kept_ref)} groups complete, {nf} of {len(pages)} page ids reclaimed")
    assert nf == len(want) and np.array_equal(free[:nf], want) and (free[nf:] == -1).all()


def test_stream_read_reads_every_word():
    """The streaming-read reference touches every 16-byte word exactly once:
    the sum of its per-wavefront partial sums equals the buffer's sum (small
    integers, exact in float32 at this size), with a ragged tail."""
    B = _b()
    n = (1 << 20) + 12                       # floats: 16-byte words plus a partial grid stride
    x = (torch.arange(n, dtype=torch.int64, device=DEV) % 7).to(torch.float32)
    sink = torch.zeros(8192, dtype=torch.float32, device=DEV)
    B.darts_stream_read(x, sink)
    torch.cuda.synchronize()
    assert float(sink.double().sum().item()) == float(x.double().sum().item())

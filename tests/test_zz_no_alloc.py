"""The allocation-free decode attention (darts_attn_decode_noalloc) through the
C ABI: two calls in a row, the second smaller, each bitwise equal to
darts_attn_decode with a caller workspace on the same inputs (ragged
contexts with chunked rows, then the equal-context decode form), one f32
call, and the size check that rejects a workspace beyond the library's
array before anything is launched."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import sweep as OS
from workload.gen import sweep_page_table

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _b():
    from paper_2605_30859_amd import binding
    binding.load_library()
    return binding


def _inputs(B, rows, hq, hkv, hd, ctx, dt, tdt, seed):
    rng = np.random.default_rng(seed)
    pt, n_pages = sweep_page_table(ctx, 16, rng, spare=3)
    q = torch.empty(rows * hq * hd, dtype=tdt, device=DEV)
    kp = torch.empty(n_pages * hkv * 16 * hd, dtype=tdt, device=DEV)
    vp = torch.empty_like(kp)
    B.darts_fill_uniform(q, OS.T_Q, seed, dt)
    B.darts_fill_kv_pool(kp, vp, n_pages, hkv, hd, seed, dt)
    return q, kp, vp, n_pages, torch.from_numpy(pt).to(DEV), torch.from_numpy(ctx.astype(np.int32)).to(DEV)


def _both(rows, hq, hkv, hd, ctx, dtype, seed, equal):
    """(noalloc output, workspace output) on the same inputs."""
    B = _b()
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dt = B.DARTS_BF16 if dtype == "bf16" else B.DARTS_F32
    q, kp, vp, n_pages, ptd, ctxd = _inputs(B, rows, hq, hkv, hd, ctx, dt, tdt, seed)
    max_ctx = int(ctx.max())
    cl = None if equal else ctxd
    a = torch.full((rows * hq * hd,), float("nan"), dtype=tdt, device=DEV)
    b = torch.full((rows * hq * hd,), float("nan"), dtype=tdt, device=DEV)
    say(f"noalloc: {dtype} rows={rows} hq={hq} hkv={hkv} hd={hd} max_ctx={max_ctx} equal={equal}")
    B.darts_attn_decode_noalloc(q, kp, vp, n_pages, ptd, cl, hq, hkv, hd, max_ctx, dt, a, n_rows=rows)
    ws = torch.empty(B.darts_attn_workspace_bytes(rows, hq, hkv, hd, max_ctx), dtype=torch.uint8, device=DEV)
    B.darts_attn_decode(q, kp, vp, n_pages, ptd, cl, hq, hkv, hd, max_ctx, dt, b, ws, n_rows=rows)
    torch.cuda.synchronize()
    return a.view(torch.int16 if dtype == "bf16" else torch.int32).cpu().numpy(), \
        b.view(torch.int16 if dtype == "bf16" else torch.int32).cpu().numpy()


def test_noalloc_two_calls_match_workspace_entry():
    B = _b()
    rng = np.random.default_rng(5)
    # first call: 192 ragged rows up to 6000 keys (rows split into chunks,
    # combined); its workspace is most of the library's array
    ctx1 = np.clip(np.rint(1500 * np.exp(rng.standard_normal(192))), 1, 6000).astype(np.int64)
    need = B.darts_attn_workspace_bytes(192, 32, 8, 128, int(ctx1.max()))
    assert need <= B.ATTN_NOALLOC_SCRATCH_BYTES
    a, b = _both(192, 32, 8, 128, ctx1, "bf16", 11, equal=False)
    assert np.array_equal(a, b)
    # second call, smaller: the equal-context decode form over 40 rows
    ctx2 = np.full(40, 777, dtype=np.int64)
    a, b = _both(40, 32, 8, 128, ctx2, "bf16", 12, equal=True)
    assert np.array_equal(a, b)
    # a float32 call with other head shapes
    ctx3 = np.array([1, 16, 17, 300, 45], dtype=np.int64)
    a, b = _both(5, 8, 2, 64, ctx3, "f32", 13, equal=False)
    assert np.array_equal(a, b)


def test_noalloc_rejects_workspace_beyond_its_array():
    """1024 rows with contexts up to 32768 need about 270 MB of workspace: the
    call is refused on the host with DARTS_EINVAL and launches nothing."""
    B = _b()
    rows, hq, hkv, hd, max_ctx = 1024, 32, 8, 128, 32768
    assert B.darts_attn_workspace_bytes(rows, hq, hkv, hd, max_ctx) > B.ATTN_NOALLOC_SCRATCH_BYTES
    q = torch.zeros(rows * hq * hd, dtype=torch.bfloat16, device=DEV)
    kp = torch.zeros(16 * hkv * 16 * hd, dtype=torch.bfloat16, device=DEV)
    pt = torch.zeros((rows, max_ctx // 16), dtype=torch.int32, device=DEV)
    out = torch.zeros_like(q)
    with pytest.raises(B.DartsError) as e:
        B.darts_attn_decode_noalloc(q, kp, kp, 16, pt, None, hq, hkv, hd, max_ctx, B.DARTS_BF16, out,
                                    n_rows=rows)
    assert e.value.status == B.DARTS_EINVAL

"""Dense projection GEMM parity (darts_gemm) against float64 products of the
same bf16 operands, over the decode batch sizes of a rollout (1 .. 512 rows,
prefill-sized M) and the decoder shapes, for every epilogue."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda"

from workload.gen import bf16_bits_from_f32, f32_from_bf16_bits


def _b():
    from paper_2605_30859_amd import binding
    binding.load_library()
    return binding


def silu(x):
    return x / (1.0 + np.exp(-x))


def _mk(rng, rows, cols, scale):
    bits = bf16_bits_from_f32((rng.standard_normal((rows, cols)) * scale).astype(np.float32))
    return bits, f32_from_bf16_bits(bits).astype(np.float64)


def _run(M, N, K, epi, seed=0, sample_rows=None):
    B = _b()
    rng = np.random.default_rng(seed + M * 7 + N + K)
    ab, a = _mk(rng, M, K, 1.0)
    wb, w = _mk(rng, N, K, 1.0 / np.sqrt(K))
    at = torch.from_numpy(ab.view(np.int16)).to(DEV)
    wt = torch.from_numpy(wb.view(np.int16)).to(DEV)
    if epi == 3:
        out = torch.zeros((M, N // 2), dtype=torch.int16, device=DEV)
    elif epi == 1:
        out = torch.zeros((M, N), dtype=torch.int16, device=DEV)
    else:
        init = rng.standard_normal((M, N)).astype(np.float32) if epi == 2 else np.zeros((M, N), np.float32)
        out = torch.from_numpy(init.copy()).to(DEV)
    wsb = B.darts_gemm_workspace_bytes(M, N, K)
    ws = torch.empty(max(wsb, 256), dtype=torch.uint8, device=DEV)
    B.darts_gemm(at, wt, out, M, N, K, B.DARTS_BF16, epi, ws)
    torch.cuda.synchronize()
    rows = np.arange(M) if sample_rows is None else np.unique(np.clip(sample_rows, 0, M - 1))
    ref = a[rows] @ w.T
    if epi == 3:
        got = f32_from_bf16_bits(out.cpu().numpy().view(np.uint16)[rows]).astype(np.float64)
        g = ref[:, [(c >> 4) * 32 + (c & 15) for c in range(N // 2)]]
        u = ref[:, [(c >> 4) * 32 + 16 + (c & 15) for c in range(N // 2)]]
        exp = silu(g) * u
        tol = 2 ** -7
    elif epi == 1:
        got = f32_from_bf16_bits(out.cpu().numpy().view(np.uint16)[rows]).astype(np.float64)
        exp = ref
        tol = 2 ** -7
    else:
        got = out.cpu().numpy()[rows].astype(np.float64)
        exp = ref + (init[rows] if epi == 2 else 0.0)
        tol = 1e-4
    scale = np.maximum(np.abs(exp).max(axis=1, keepdims=True), 1e-3)
    err = (np.abs(got - exp) / scale).max()
    assert err <= tol, (M, N, K, epi, err)


@pytest.mark.parametrize("M", [1, 5, 16, 17, 33, 64, 65, 100, 128, 129, 200, 256, 300, 512])
def test_gemm_qkv_shape_all_batch_sizes(M):
    print(f"gemm M={M}", flush=True)
    _run(M, 6144, 4096, 0)


@pytest.mark.parametrize("M,N,K,epi", [(512, 4096, 4096, 2), (37, 4096, 4096, 2),
                                       (512, 24576, 4096, 3), (9, 24576, 4096, 3), (130, 24576, 4096, 3),
                                       (512, 4096, 12288, 2), (3, 4096, 12288, 2), (200, 4096, 12288, 2),
                                       (64, 1536, 1024, 1), (300, 32000, 1024, 0), (1024, 5120, 2048, 0),
                                       # small-batch exact-fill tiles (64 and 128 rows, 64 and 96 wide),
                                       # every epilogue, with and without a K split
                                       (64, 4096, 4096, 2), (100, 4096, 4096, 2), (16, 4096, 12288, 2),
                                       (64, 4096, 12288, 2), (50, 24576, 4096, 3), (128, 24576, 4096, 3),
                                       (60, 6144, 4096, 1), (97, 6144, 4096, 1), (40, 8192, 1024, 3),
                                       (33, 2048, 4096, 2),
                                       # the Qwen3-30B-A3B attention projections (QKV, O with the
                                       # residual add) at 100-513 rows, with and without a K split
                                       (128, 5120, 2048, 0), (200, 5120, 2048, 0), (354, 5120, 2048, 0),
                                       (513, 5120, 2048, 0), (100, 2048, 4096, 2), (200, 2048, 4096, 2),
                                       (256, 2048, 4096, 2), (354, 2048, 4096, 2), (512, 2048, 4096, 2)])
def test_gemm_decoder_shapes(M, N, K, epi):
    print(f"gemm M={M} N={N} K={K} epi={epi}", flush=True)
    _run(M, N, K, epi)


def test_gemm_lm_head_full_size_sampled_rows():
    """LM head at the Qwen3-8B shape (151936 x 4096), 512 rows; sampled rows."""
    _run(512, 151936, 4096, 0, sample_rows=np.array([0, 1, 63, 64, 255, 256, 300, 511]))


def test_gemm_prefill_size_sampled_rows():
    """Prefill-sized M (32 prompts x 512 tokens) on the QKV shape; sampled rows."""
    _run(16384, 6144, 4096, 0, sample_rows=np.array([0, 1, 127, 128, 8191, 16000, 16383]))

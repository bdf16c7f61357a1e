"""Host-side argument checks of the stateless entries (no GPU needed: every
call here returns before any device work).  A zero-size call is a no-op
returning DARTS_OK with NULL device pointers; bad scalars give DARTS_EINVAL."""
import ctypes as C

import pytest

from paper_2605_30859_amd import binding as B

OK, EINVAL = B.DARTS_OK, B.DARTS_EINVAL
N = None


@pytest.fixture(scope="module")
def lib():
    return B.load_library()


def test_zero_size_calls_are_noops(lib):
    # attention: 0 rows, Qwen3-8B heads
    assert lib.darts_attn_decode(N, N, N, 1, N, 1, N, 0, 32, 8, 128, 16, B.DARTS_BF16, N, N, 0, N) == OK
    assert lib.darts_attn_decode_shared(N, N, N, 4, N, 4, 1, N, 16, 2, 48, 0, 32, 8, 128,
                                        B.DARTS_BF16, N, N, 0, N) == OK
    assert lib.darts_sample(N, 0, 151936, B.DARTS_BF16, 1, N, N, 1.0, N, N, N, N, N) == OK
    assert lib.darts_gemm(N, N, N, 0, 4096, 4096, B.DARTS_BF16, 0, N, 0, N) == OK
    assert lib.darts_select_groups(N, N, N, 0, 16, 8, 1, 16, 1, N, N, N, N, N, N, N, N) == OK
    assert lib.darts_group_advantages(N, 0, 8, N, 0, C.c_float(1e-6), N, N) == OK
    assert lib.darts_stream_read(N, 0, N, N) == OK
    assert lib.darts_debug_gumbel(N, N, 0, N) == OK
    assert lib.darts_debug_gumbel_fast(N, N, 0, N) == OK


def test_bad_scalars_are_rejected(lib):
    bf = B.DARTS_BF16
    # attention: unsupported head_dim, GQA ratio > 16, page table narrower than max_ctx
    assert lib.darts_attn_decode(N, N, N, 1, N, 1, N, 0, 32, 8, 48, 16, bf, N, N, 0, N) == EINVAL
    assert lib.darts_attn_decode(N, N, N, 1, N, 1, N, 0, 64, 2, 128, 16, bf, N, N, 0, N) == EINVAL
    assert lib.darts_attn_decode(N, N, N, 1, N, 1, N, 0, 32, 8, 128, 17, bf, N, N, 0, N) == EINVAL
    assert lib.darts_attn_decode(N, N, N, 1, N, 1, N, -1, 32, 8, 128, 16, bf, N, N, 0, N) == EINVAL
    # sampler: vocabulary not a multiple of 4, non-positive temperature, unknown dtype
    assert lib.darts_sample(N, 0, 6, bf, 1, N, N, 1.0, N, N, N, N, N) == EINVAL
    assert lib.darts_sample(N, 0, 8, bf, 1, N, N, 0.0, N, N, N, N, N) == EINVAL
    assert lib.darts_sample(N, 0, 8, 7, 1, N, N, 1.0, N, N, N, N, N) == EINVAL
    # rows but no buffers
    assert lib.darts_sample(N, 3, 8, bf, 1, N, N, 1.0, N, N, N, N, N) == EINVAL
    # gemm: bf16 shapes must tile (N % 128, K % 256); SwiGLU needs N % 32
    assert lib.darts_gemm(N, N, N, 0, 4000, 4096, bf, 0, N, 0, N) == EINVAL
    assert lib.darts_gemm(N, N, N, 0, 4096, 1000, bf, 0, N, 0, N) == EINVAL
    assert lib.darts_gemm(N, N, N, 0, 48, 64, B.DARTS_F32, 3, N, 0, N) == EINVAL
    assert lib.darts_gemm(N, N, N, 1, 4096, 4096, bf, 0, N, 0, N) == EINVAL
    # selection: k > m, m > 64, trajectories not whole groups, dual-end with L >= k
    assert lib.darts_select_groups(N, N, N, 0, 8, 9, 1, 16, 1, N, N, N, N, N, N, N, N) == EINVAL
    assert lib.darts_select_groups(N, N, N, 0, 65, 8, 1, 16, 1, N, N, N, N, N, N, N, N) == EINVAL
    assert lib.darts_select_groups(N, N, N, 17, 16, 8, 1, 16, 1, N, N, N, N, N, N, N, N) == EINVAL
    assert lib.darts_select_groups(N, N, N, 0, 12, 8, 8, 16, 1, N, N, N, N, N, N, N, N) == EINVAL
    # selection with page reclaim: page lists without the output, count or scratch buffers
    D = C.c_void_p(256)          # never dereferenced: the call fails its argument check first
    assert lib.darts_select_groups(D, D, D, 16, 16, 8, 1, 16, 1, D, D, D, D, N, D, D, N) == EINVAL
    assert lib.darts_select_groups(D, D, D, 16, 16, 8, 1, 16, 1, D, D, D, D, D, D, N, N) == EINVAL
    # streaming read: not whole 16-byte words
    assert lib.darts_stream_read(N, 24, N, N) == EINVAL


def test_attention_equal_contexts_arguments(lib):
    # NULL contexts (every row has max_ctx keys) pass the checks; with rows
    # present a NULL q is still rejected before any device work
    bf = B.DARTS_BF16
    assert lib.darts_attn_decode(N, N, N, 1, N, 1, N, 0, 32, 8, 128, 16, bf, N, N, 0, N) == OK
    assert lib.darts_attn_decode(N, N, N, 1, N, 1, N, 4, 32, 8, 128, 16, bf, N, N, 0, N) == EINVAL
    # the binding needs the row count when no contexts are given
    with pytest.raises(ValueError):
        B.darts_attn_decode(None, None, None, 1, None, None, 32, 8, 128, 16, bf, None, None)


def test_context_calls_reject_a_null_context(lib):
    assert lib.darts_debug_fill_kv(N, 0xFF) == EINVAL
    assert lib.darts_debug_logits(N, N, N) == EINVAL

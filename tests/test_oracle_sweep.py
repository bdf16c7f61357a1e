"""Pins for the kernel-sweep oracle (oracle/sweep.py) and the two margin
functions that decide which near-tie rows a parity test may excuse
(oracle.sampler.top2_margin, oracle.model.route_margin).

* sweep_values: the float64 value of each Philox word's mapping, rounded to
  bfloat16 by PyTorch's own conversion (round to nearest even), from words the
  block generator produces (both generators are pinned to the published
  Philox4x32-10 vectors).
* attention_row: the paged layout gathered independently (the whole pool
  generated first, then indexed by page table row and slot) and passed to
  oracle.model.attention, which is pinned to PyTorch's scaled dot-product
  attention with grouped-query heads; G = 1, 4 and 8 query heads per kv head,
  ragged contexts and partly filled last pages; one key returns its value;
  equal keys give the mean of the values.
* top2_margin: brute force over all index pairs on small vocabularies,
  including constructed exact ties (margin 0).
* route_margin: a hand-worked example with a tie between ranks k and k+1.
"""
import math
from types import SimpleNamespace

import numpy as np
import pytest
import torch

from oracle import model as M
from oracle import sweep as OS
from oracle.philox import philox_range
from oracle.sampler import perturbed_scores, top2_margin


def test_sweep_values_map_and_rounding():
    seed, tensor, n = 1, OS.T_K, 4096
    words = philox_range(0, n, tensor, 0, OS.TAG_SWEEP, seed).astype(np.float64)
    exact = (np.floor(words / 256.0) * 1.0 + (np.floor(words / 256.0) % 2 == 0)) * 2.0 ** -23 - 1.0
    want = torch.tensor(exact, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    got = OS.sweep_values(tensor, np.arange(n, dtype=np.uint64), seed)
    np.testing.assert_array_equal(got, want)
    # bf16 rounding can reach +-1 exactly
    assert (np.abs(got) <= 1).all() and abs(got.mean()) < 0.05 and abs(got.var() - 1 / 3) < 0.02


def _pool(seed, n_pages, hkv, hd, tensor):
    """Whole pool [page][kv head][slot][hd] in the logical layout."""
    idx = np.arange(n_pages * hkv * 16 * hd, dtype=np.uint64)
    return OS.sweep_values(tensor, idx, seed).reshape(n_pages, hkv, 16, hd)


@pytest.mark.parametrize("hq,hkv,hd", [(4, 4, 32), (8, 2, 64), (16, 2, 32)])
def test_attention_row_equals_gathered_definition(hq, hkv, hd):
    seed = 5
    ctxs = [1, 16, 17, 45]
    n_pages = 12
    rng = np.random.default_rng(0)
    Kp, Vp = _pool(seed, n_pages, hkv, hd, OS.T_K), _pool(seed, n_pages, hkv, hd, OS.T_V)
    for row, ctx in enumerate(ctxs):
        pt = rng.permutation(n_pages)[: -(-ctx // 16)]
        q = OS.sweep_values(OS.T_Q, np.arange(row * hq * hd, (row + 1) * hq * hd, dtype=np.uint64),
                            seed).reshape(hq, hd)
        j = np.arange(ctx)
        K = Kp[pt[j // 16], :, j % 16, :]
        V = Vp[pt[j // 16], :, j % 16, :]
        want = M.attention(q, K, V, hkv)
        got = OS.attention_row(row, ctx, pt, seed, hq, hkv, hd)
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-13)
        if ctx == 1:      # one key: the output is that key's value for every head
            for h in range(hq):
                np.testing.assert_allclose(got[h], V[0, (h * hkv) // hq], rtol=0, atol=1e-15)


def test_attention_definition_special_cases():
    """Equal keys: softmax is uniform and the output is the mean of the values;
    GQA with G heads per kv head equals MHA with each kv head repeated G times."""
    rng = np.random.default_rng(2)
    hq, hkv, hd, ctx = 8, 2, 16, 9
    q = rng.standard_normal((hq, hd))
    K = np.repeat(rng.standard_normal((1, hkv, hd)), ctx, axis=0)
    V = rng.standard_normal((ctx, hkv, hd))
    out = M.attention(q, K, V, hkv)
    for h in range(hq):
        np.testing.assert_allclose(out[h], V[:, (h * hkv) // hq].mean(axis=0), rtol=0, atol=1e-14)
    K = rng.standard_normal((ctx, hkv, hd))
    np.testing.assert_allclose(M.attention(q, K, V, hkv),
                               M.attention(q, np.repeat(K, hq // hkv, axis=1), np.repeat(V, hq // hkv, axis=1),
                                           hq), rtol=0, atol=1e-14)


def _brute_margin(sc):
    best = max(range(len(sc)), key=lambda i: (float(sc[i]), -i))
    second = max(float(sc[j]) for j in range(len(sc)) if j != best)
    return float(sc[best]) - second


def test_top2_margin_brute_force_and_ties():
    rng = np.random.default_rng(8)
    for trial in range(200):
        V = int(rng.integers(2, 17))
        z = (rng.normal(0, 2, V)).astype(np.float32)
        sc = perturbed_scores(z, 1.0, trial, 3, 99)
        assert top2_margin(z, 1.0, trial, 3, 99) == pytest.approx(_brute_margin(sc), abs=0)
    # constructed exact tie: adjust entry 1 until its perturbed score equals entry 0's
    z = np.full(6, -30.0, dtype=np.float32)
    z[:2] = 0.0
    sc = perturbed_scores(z, 1.0, 7, 0, 99)
    z[1] = np.float32(sc[0] - sc[1])
    for _ in range(64):
        s1 = perturbed_scores(z, 1.0, 7, 0, 99)
        if s1[1] == s1[0]:
            break
        z[1] = np.nextafter(z[1], np.float32(np.inf) if s1[1] < s1[0] else np.float32(-np.inf))
    s1 = perturbed_scores(z, 1.0, 7, 0, 99)
    assert s1[1] == s1[0] and s1[0] == s1.max()
    assert top2_margin(z, 1.0, 7, 0, 99) == 0.0


def test_route_margin_hand_example():
    p = np.array([[0.3, 0.25, 0.25, 0.2], [0.1, 0.6, 0.05, 0.25]])
    cfg = lambda k: SimpleNamespace(top_k=k)
    assert list(M.route_margin(cfg(2), p)) == [0.0, pytest.approx(0.15)]
    assert list(M.route_margin(cfg(1), p)) == [pytest.approx(0.05), pytest.approx(0.35)]
    assert list(M.route_margin(cfg(3), p)) == [pytest.approx(0.05), pytest.approx(0.05)]
    assert np.isinf(M.route_margin(cfg(4), p)).all()

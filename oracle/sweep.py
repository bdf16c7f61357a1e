"""Kernel-sweep data and per-row decode attention (definition).

Sweep tensors are Philox-filled so that both sides can produce them without
sharing data: element idx of tensor t is
    bf16( ((w >> 8) | 1) * 2^-23 - 1 ),  w = Philox(key=seed, counter=(idx>>2, t, 0, TAG_SWEEP)) word idx&3
with logical layouts  Q: [rows][Hq][hd],  K and V pools: [page][Hkv][slot][hd].

Decode attention for one row (definition, float64):
    out[h] = sum_j softmax_j(q_h . k_j / sqrt(hd)) v_j   over the row's ctx keys,
    key j lives in page table[j // page_size], slot j % page_size, kv head floor(h*Hkv/Hq).
Pinned (tests/test_oracle_sweep.py): sweep_values against the word mapping
evaluated in float64 and rounded by PyTorch's bfloat16 conversion;
attention_row against the paged pool gathered independently and passed to
oracle.model.attention (itself pinned to PyTorch's grouped-query
scaled dot-product attention), for 1, 4 and 8 query heads per kv head,
ragged contexts and partly filled last pages; one key returns its value.
"""
import math

import numpy as np

from .philox import philox_words
from .model import round_bf16

TAG_SWEEP = 3
T_Q, T_K, T_V = 0, 1, 2


def sweep_values(tensor, idx, seed):
    w = philox_words(np.asarray(idx, dtype=np.uint64), tensor, 0, TAG_SWEEP, seed)
    k = ((w >> np.uint32(8)) | np.uint32(1)).astype(np.float32)
    v = (k * np.float32(2.0 ** -23) - np.float32(1.0)).astype(np.float32)
    return round_bf16(v).astype(np.float64)


def attention_row(row, ctx, pt_row, seed, hq, hkv, hd, page=16):
    """Attention output [hq, hd] of sweep row ``row`` (float64)."""
    q = sweep_values(T_Q, np.arange(row * hq * hd, (row + 1) * hq * hd, dtype=np.uint64), seed)
    q = q.reshape(hq, hd)
    j = np.arange(ctx)
    pg = np.asarray(pt_row, dtype=np.int64)[j // page]
    slot = j % page
    # element index for (page, kv head, slot, dim)
    base = ((pg[:, None] * hkv + np.arange(hkv)[None, :]) * page + slot[:, None]) * hd   # [ctx, hkv]
    idx = (base[:, :, None] + np.arange(hd)[None, None, :]).astype(np.uint64)
    K = sweep_values(T_K, idx.ravel(), seed).reshape(ctx, hkv, hd)
    V = sweep_values(T_V, idx.ravel(), seed).reshape(ctx, hkv, hd)
    out = np.empty((hq, hd))
    for h in range(hq):
        kh = (h * hkv) // hq
        s = K[:, kh, :] @ q[h] / math.sqrt(hd)
        s -= s.max()
        p = np.exp(s)
        p /= p.sum()
        out[h] = p @ V[:, kh, :]
    return out

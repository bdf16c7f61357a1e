"""Philox4x32-10 counter-based generator (Salmon, Moraes, Dror, Shaw, SC'11,
"Parallel random numbers: as easy as 1, 2, 3").

Written from the published definition: a 4x32-bit counter block and a 2x32-bit
key; each of the 10 rounds multiplies words 0 and 2 by the two round
multipliers (0xD2511F53, 0xCD9E8D57), keeping the high and low 32-bit halves,
permutes the words and XORs the high halves with the other counter words and
the round key; the key is bumped by the Weyl constants (0x9E3779B9,
0xBB67AE85) between rounds.

Pinned by the published known-answer vectors (tests/golden/philox4x32_10_kat.txt).
"""
import numpy as np

_M0 = np.uint64(0xD2511F53)
_M1 = np.uint64(0xCD9E8D57)
_W0 = np.uint64(0x9E3779B9)
_W1 = np.uint64(0xBB67AE85)
_MASK = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Vectorised Philox4x32-10.  Counter words / key words are broadcastable
    integer arrays (values < 2^32).  Returns four uint32 arrays."""
    x0 = np.asarray(c0, dtype=np.uint64) & _MASK
    x1 = np.asarray(c1, dtype=np.uint64) & _MASK
    x2 = np.asarray(c2, dtype=np.uint64) & _MASK
    x3 = np.asarray(c3, dtype=np.uint64) & _MASK
    x0, x1, x2, x3 = np.broadcast_arrays(x0, x1, x2, x3)
    key0 = np.uint64(int(k0) & 0xFFFFFFFF)
    key1 = np.uint64(int(k1) & 0xFFFFFFFF)
    for r in range(10):
        if r > 0:
            key0 = (key0 + _W0) & _MASK
            key1 = (key1 + _W1) & _MASK
        p0 = _M0 * x0            # < 2^64, exact in uint64
        p1 = _M1 * x2
        hi0, lo0 = p0 >> _S32, p0 & _MASK
        hi1, lo1 = p1 >> _S32, p1 & _MASK
        x0, x1, x2, x3 = hi1 ^ x1 ^ key0, lo1, hi0 ^ x3 ^ key1, lo0
    return (x0.astype(np.uint32), x1.astype(np.uint32),
            x2.astype(np.uint32), x3.astype(np.uint32))


def philox_range(start, n, c1, c2, c3, seed):
    """philox_words(arange(start, start + n), ...) for scalar c1, c2, c3 and a
    start that is a multiple of 4: each counter block is evaluated once and its
    four words are laid out in order (the same values, fewer evaluations)."""
    assert start % 4 == 0
    nb = (n + 3) // 4
    blk = np.arange(start // 4, start // 4 + nb, dtype=np.uint64)
    seed = int(seed)
    w = philox4x32_10(blk, c1, c2, c3, seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    return np.stack(w, axis=1).reshape(-1)[:n].astype(np.uint32)


def philox_words(idx, c1, c2, c3, seed):
    """Word ``idx & 3`` of Philox(counter=(idx >> 2, c1, c2, c3), key=(seed lo, seed hi))."""
    idx = np.asarray(idx, dtype=np.uint64)
    blk = idx >> np.uint64(2)
    sel = (idx & np.uint64(3)).astype(np.int64)
    seed = int(seed)
    w = philox4x32_10(blk, c1, c2, c3, seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    out = np.choose(sel, w)
    return out.astype(np.uint32)


def u24_odd(words):
    """Map a 32-bit word to u = ((w >> 8) | 1) * 2^-24, an exact float32 in (0, 1)."""
    w = np.asarray(words, dtype=np.uint32)
    k = ((w >> np.uint32(8)) | np.uint32(1)).astype(np.float32)
    return (k * np.float32(2.0 ** -24)).astype(np.float32)

"""Natural logarithm and the Gumbel map as an exact float32 operation sequence.

The sampled token is an argmax over float32 perturbed scores, so both sides
must produce bit-identical Gumbel noise.  The logarithm is therefore defined
here as a fixed sequence of IEEE float32 operations (each correctly rounded,
no fused multiply-add), following the classical atanh-series method:

    x = 2^e * m,  m in (sqrt(1/2), sqrt(2)]
    t = (m - 1) / (m + 1)            [computed as f / (2 + f), f = m - 1]
    ln m = 2 t (1 + t^2/3 + t^4/5 + t^6/7 + t^8/9 + t^10/11)
    ln x = e * ln2_hi + (e * ln2_lo + ln m)

with ln 2 split into a 16-bit head (so e * ln2_hi is exact) and a float32 tail.
|t| <= 0.1716, so the dropped series term is below 1e-9 relative.

Gumbel noise: g(u) = -ln(-ln(u)) for u = ((w >> 8) | 1) * 2^-24 in (0, 1).

Pinned by: agreement with the float64 library logarithm to a few ulp over all
2^23 possible u and all 2^23 values -ln(u) (tests/test_oracle_sampler.py), and
by a chi-square test of the Gumbel-max token frequencies against softmax.
"""
import numpy as np

F = np.float32
_LN2_HI = F(45426.0 / 65536.0)                                # 16 significant bits
_LN2_LO = F(0.6931471805599453094 - 45426.0 / 65536.0)        # rounded tail
_SQRT2 = F(1.4142135623730951)
_C3, _C5, _C7, _C9, _C11 = F(1 / 3), F(1 / 5), F(1 / 7), F(1 / 9), F(1 / 11)


def ln_f32(x):
    """Own natural log of positive, finite, normal float32 values (array)."""
    x = np.asarray(x, dtype=np.float32)
    bits = x.view(np.uint32)
    e = ((bits >> np.uint32(23)) & np.uint32(0xFF)).astype(np.int32) - 127
    mbits = (bits & np.uint32(0x007FFFFF)) | np.uint32(0x3F800000)
    m = mbits.view(np.float32)
    big = m > _SQRT2
    m = np.where(big, m * F(0.5), m).astype(np.float32)   # exact halving
    e = np.where(big, e + 1, e)
    f = (m - F(1.0)).astype(np.float32)                    # exact (Sterbenz)
    den = (F(2.0) + f).astype(np.float32)
    t = (f / den).astype(np.float32)
    t2 = (t * t).astype(np.float32)
    p = np.full_like(t, _C11)
    for c in (_C9, _C7, _C5, _C3, F(1.0)):
        p = (p * t2).astype(np.float32)
        p = (p + c).astype(np.float32)
    lnm = ((t + t).astype(np.float32) * p).astype(np.float32)
    ef = e.astype(np.float32)
    lo = (ef * _LN2_LO).astype(np.float32)
    lo = (lo + lnm).astype(np.float32)
    hi = (ef * _LN2_HI).astype(np.float32)
    return (hi + lo).astype(np.float32)


def gumbel_f32(u):
    """g(u) = -ln(-ln u) with the float32 operation sequence above."""
    u = np.asarray(u, dtype=np.float32)
    a = (-ln_f32(u)).astype(np.float32)
    return (-ln_f32(a)).astype(np.float32)

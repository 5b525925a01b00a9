"""The fixed-point limb split the probe's MFMA logits rest on, checked on the
CPU with exact integer / rational arithmetic (no GPU, neither the oracle nor
the HIP library involved).

For a vector x of bf16 values with E = floor(log2 max|x_i|) and F = E - 13:
n_i = trunc(x_i 2^-F) satisfies |n_i| < 2^14 and splits into a low limb
n_i & 127 in [0, 127] and a high limb n_i >> 7 in [-128, 127]; x_g = 2^F n
and x_r = x - x_g are exact, x_r is bf16-representable, and for two vectors
the four int8 limb dot products give
  <q_g, k_g> = 2^(Fq + Fk) (P00 + 2^7 (P01 + P10) + 2^14 P11)
exactly, each P within int32, so <q, k> = that + <q_r, k> + <q_g, k_r>.
Elements at or above 2^-6 of the vector's maximum have x_r = 0.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

FRAC_BITS = 13


def bf16_values(rng, n, exp_lo, exp_hi, zero_frac=0.0):
    """n random bf16 numbers (as Python floats) with binary exponents drawn in
    [exp_lo, exp_hi] (subnormals included below -126), random signs and
    8-bit significands, and a fraction of +-0."""
    out = []
    for _ in range(n):
        if rng.random() < zero_frac:
            out.append(-0.0 if rng.random() < 0.5 else 0.0)
            continue
        e = int(rng.integers(exp_lo, exp_hi + 1))
        if e < -126:                                  # bf16 subnormal: m 2^-133, m < 128
            m = int(rng.integers(1, 128))
            v = m * 2.0 ** -133
        else:
            m = int(rng.integers(128, 256))           # 8-bit significand
            v = m * 2.0 ** (e - 7)
        out.append(-v if rng.random() < 0.5 else v)
    return out


def is_bf16(v: float) -> bool:
    if v == 0.0 or math.isinf(v):
        return True
    u = np.float32(v).view(np.uint32)
    return float(np.float32(v)) == v and (int(u) & 0xFFFF) == 0


def split(x):
    amax = max(abs(v) for v in x)
    F = (math.frexp(amax)[1] - 1 - FRAC_BITS) if amax > 0 else 0
    n = [int(math.trunc(math.ldexp(v, -F))) for v in x]
    g = [math.ldexp(k, F) for k in n]
    r = [v - gv for v, gv in zip(x, g)]
    return F, n, g, r


def limbs(n):
    lo = [k & 127 for k in n]
    hi = [k >> 7 for k in n]
    return lo, hi


SPANS = [(-3, 2), (-20, 3), (-40, 4), (-133, -120), (-133, 10), (100, 127), (-8, -8)]


@pytest.mark.parametrize("span", SPANS)
@pytest.mark.parametrize("zeros", [0.0, 0.3])
def test_split_is_exact_and_bounded(span, zeros):
    rng = np.random.default_rng(abs(hash((span, zeros))) % (2 ** 32))
    for _ in range(20):
        x = bf16_values(rng, 128, *span, zero_frac=zeros)
        F, n, g, r = split(x)
        assert all(-2 ** 14 < k < 2 ** 14 for k in n)
        lo, hi = limbs(n)
        assert all(0 <= a <= 127 for a in lo) and all(-128 <= b <= 127 for b in hi)
        assert all(b * 128 + a == k for a, b, k in zip(lo, hi, n))
        for v, gv, rv in zip(x, g, r):
            assert Fraction(gv) + Fraction(rv) == Fraction(v)     # exact
            assert is_bf16(rv) and is_bf16(gv)
            assert abs(rv) < 2.0 ** F                           # below the grid step
        amax = max(abs(v) for v in x)
        for v, rv in zip(x, r):                                 # on the grid from 2^-6 max
            if abs(v) >= amax * 2.0 ** -6:
                assert rv == 0.0


@pytest.mark.parametrize("sq,sk", [(SPANS[0], SPANS[1]), (SPANS[2], SPANS[0]),
                                   (SPANS[3], SPANS[4]), (SPANS[5], SPANS[6]),
                                   (SPANS[1], SPANS[1])])
def test_limb_dot_products_are_exact(sq, sk):
    rng = np.random.default_rng(7)
    for _ in range(10):
        q = bf16_values(rng, 128, *sq, zero_frac=0.1)
        k = bf16_values(rng, 128, *sk, zero_frac=0.1)
        Fq, nq, gq, rq = split(q)
        Fk, nk, gk, rk = split(k)
        ql, qh = limbs(nq)
        kl, kh = limbs(nk)
        p00 = sum(a * b for a, b in zip(ql, kl))
        p01 = sum(a * b for a, b in zip(ql, kh))
        p10 = sum(a * b for a, b in zip(qh, kl))
        p11 = sum(a * b for a, b in zip(qh, kh))
        assert all(abs(p) < 2 ** 31 for p in (p00, p01, p10, p11))
        x = p00 + (p01 + p10) * 128
        assert abs(x) < 2 ** 30                                 # the kernel's int32 sum
        T = x + p11 * 2 ** 14
        assert abs(T) < 2 ** 36 and float(T) == T               # exact in binary64
        exact_g = sum(Fraction(a) * Fraction(b) for a, b in zip(gq, gk))
        assert Fraction(T) * Fraction(2) ** (Fq + Fk) == exact_g
        # the full dot product: grid part plus the two residual products
        exact = sum(Fraction(a) * Fraction(b) for a, b in zip(q, k))
        resid = (sum(Fraction(a) * Fraction(b) for a, b in zip(rq, k)) +
                 sum(Fraction(a) * Fraction(b) for a, b in zip(gq, rk)))
        assert exact_g + resid == exact
        # the bound that decides whether the residual product is formed
        bound = (sum(abs(v) for v in rq) * max(abs(v) for v in k) +
                 max(abs(v) for v in q) * sum(abs(v) for v in rk))
        assert abs(resid) <= Fraction(bound)


def test_zero_and_signed_zero_vectors():
    for x in ([0.0] * 128, [-0.0] * 128, [0.0, -0.0] * 64):
        F, n, g, r = split(x)
        assert F == 0 and all(k == 0 for k in n) and all(v == 0.0 for v in r)

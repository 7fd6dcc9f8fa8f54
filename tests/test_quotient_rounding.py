"""The sigmoid surrogate's quotient in the backward kernels: a reciprocal
refined by one Newton step and two corrections by the exact residual
(mfpsn_surrogate.h, quot_1_4).  Checked here in exact rational arithmetic,
with each float operation rounded once to nearest even and the hardware
reciprocal modelled as the correctly rounded one moved by -1, 0 or +1 ulp:
for denominators in [1, 4] and numerators zero or in [2^-100, 2^62] the
result is the correctly rounded quotient, and for denominator 1 it is the
numerator for every float numerator, subnormals included.
"""
import random
from fractions import Fraction as F

import numpy as np
import pytest


def _ulp(a: F) -> F:
    a = abs(a)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if F(2) ** e > a:
        e -= 1
    return F(2) ** (max(e, -126) - 23)


def rn32(x: F) -> F:
    """x rounded to the nearest float32, ties to even (subnormals included)."""
    if x == 0:
        return F(0)
    u = _ulp(x)
    m = abs(x) / u
    fl = m.numerator // m.denominator
    rem = m - fl
    if rem > F(1, 2) or (rem == F(1, 2) and fl % 2 == 1):
        fl += 1
    return (fl * u) if x > 0 else -(fl * u)


def quot(n: F, b: F, dr: int) -> F:
    r = rn32(1 / b)
    r = r + dr * _ulp(r)
    e = rn32(1 - b * r)
    r = rn32(e * r + r)
    q = rn32(n * r)
    t = rn32(n - b * q)
    q = rn32(t * r + q)
    t = rn32(n - b * q)
    return rn32(t * r + q)


def f32(v: float) -> F:
    return F(float(np.float32(v)))


@pytest.mark.parametrize("seed", [0, 1])
def test_quotient_is_correctly_rounded(seed):
    rng = random.Random(seed)
    for it in range(600):
        if it % 2 == 0:
            den = rn32(1 + f32(rng.random()))   # (1 + e)^2 as the surrogate forms it
            b = rn32(den * den)
        else:
            b = f32(1 + 3 * rng.random())
        n = f32(2.0 ** rng.uniform(-100, 62))
        if it % 3 == 0:
            # numerators whose quotient lies next to a rounding midpoint
            q = rn32(n / b)
            n = rn32(b * (q + _ulp(q) / 2))
        want = rn32(n / b)
        for dr in (-1, 0, 1):
            assert quot(n, b, dr) == want, (float(n), float(b), dr)
        assert quot(F(0), b, 0) == 0


def test_denominator_one_returns_the_numerator():
    rng = random.Random(2)
    for _ in range(300):
        n = rn32(f32(2.0 ** rng.uniform(-149, 62)))
        for dr in (-1, 0, 1):
            assert quot(n, F(1), dr) == n

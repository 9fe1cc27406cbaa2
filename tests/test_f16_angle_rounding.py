"""The binary16 step settles sin and cos of an angle that lands next to a
binary16 rounding midpoint from binary64 values: on |theta| <= 1/4 the
Taylor polynomials of the binary64 step (through theta^13 and theta^12,
Horner form with fused multiply-adds), which must round to binary16 exactly
as the C library's binary64 sin and cos do (the oracle's definition).  The
binary16 angles in that range are few, so this checks every one of them,
emulating each fused multiply-add exactly (both functions are exactly odd
or even in that form, so the non-negative angles suffice)."""
import math
from fractions import Fraction

import numpy as np

SIN = [Fraction(1, math.factorial(13)), -Fraction(1, math.factorial(11)),
       Fraction(1, math.factorial(9)), -Fraction(1, math.factorial(7)),
       Fraction(1, math.factorial(5)), -Fraction(1, math.factorial(3))]
COS = [Fraction(1, math.factorial(12)), -Fraction(1, math.factorial(10)),
       Fraction(1, math.factorial(8)), -Fraction(1, math.factorial(6)),
       Fraction(1, math.factorial(4)), -Fraction(1, 2)]


def rn(q: Fraction) -> Fraction:
    return Fraction(q.numerator / q.denominator)  # correctly rounded to binary64


def fma(a, b, c):
    return rn(a * b + c)


def poly_sin(th: float) -> float:
    t = Fraction(th)
    z = rn(t * t)
    c = [rn(k) for k in SIN]  # coefficients as the compiler rounds 1.0 / n!
    p = c[0]
    for k in c[1:]:
        p = fma(p, z, k)
    return float(fma(rn(t * z), p, t))


def poly_cos(th: float) -> float:
    t = Fraction(th)
    z = rn(t * t)
    c = [rn(k) for k in COS]
    q = c[0]
    for k in c[1:]:
        q = fma(q, z, k)
    return float(fma(z, q, Fraction(1)))


def test_every_small_binary16_angle_rounds_like_libm():
    bits = np.arange(0, 0x3400 + 1, dtype=np.uint16)  # binary16 0 .. 0.25
    angles = bits.view(np.float16).astype(np.float64)
    assert angles[-1] == 0.25 and len(angles) == 0x3401
    bad = []
    for th in angles:
        for poly, ref in ((poly_sin, math.sin), (poly_cos, math.cos)):
            if np.float16(poly(th)) != np.float16(ref(th)):
                bad.append((th, poly.__name__))
    assert not bad, bad[:5]


def test_polynomials_within_an_ulp_of_libm():
    rng = np.random.default_rng(3)
    for th in rng.uniform(-0.25, 0.25, 2000):
        for poly, ref in ((poly_sin, math.sin), (poly_cos, math.cos)):
            assert abs(poly(th) - ref(th)) <= math.ulp(ref(th)), (th, poly.__name__)

"""The divisions by the total mass M = 1.1 in the step kernels are a
product with the rounded reciprocal corrected once with the exact residual
(Markstein's correction) instead of a division.  These CPU checks back the
claim that this gives the correctly rounded quotient:

* binary32: every finite dividend, exhaustively (a C program, ~25 s on 8
  cores); mismatches may only occur below 2^-104, where the quotient
  itself is near the subnormal range;
* binary64: exact rational arithmetic on random dividends over the whole
  exponent range that matters and on dividends built so that x / M falls
  next to a rounding midpoint (the hard cases for any division scheme).
"""
import math
import os
import random
import subprocess
from fractions import Fraction

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def test_binary32_exhaustive(tmp_path):
    exe = str(tmp_path / "division_check")
    subprocess.run(["gcc", "-O2", "-fopenmp", "-ffp-contract=off",
                    os.path.join(HERE, "division_check.c"), "-o", exe, "-lm"], check=True)
    out = subprocess.run([exe], capture_output=True, text=True, check=True, timeout=600).stdout
    count, worst = out.split()
    assert float.fromhex(worst) < 2.0 ** -104, out
    assert int(count) > 0  # the subnormal-range exceptions exist: the check really ran


def _rn(q: Fraction) -> float:
    return q.numerator / q.denominator  # int / int: correctly rounded to binary64


def _markstein64(x: float, m: float, inv: float) -> float:
    q = _rn(Fraction(x) * Fraction(inv))
    r = _rn(Fraction(x) - Fraction(q) * Fraction(m))  # fma(-q, m, x)
    return _rn(Fraction(r) * Fraction(inv) + Fraction(q))  # fma(r, inv, q)


def test_binary64_random_and_near_midpoint_dividends():
    m = 0.1 + 1.0
    inv = _rn(1 / Fraction(m))
    rng = random.Random(20260)
    xs = [rng.uniform(1, 2) * 2.0 ** rng.randint(-900, 900) * rng.choice((-1, 1))
          for _ in range(20000)]
    # dividends whose quotient lies within a few ulps of a midpoint between
    # two binary64 values
    for _ in range(20000):
        q = rng.uniform(1, 2) * 2.0 ** rng.randint(-30, 30)
        half_ulp = Fraction(2) ** (math.frexp(q)[1] - 54)  # q in [2^(e-1), 2^e): ulp 2^(e-53)
        mid = Fraction(q) + half_ulp
        xs.append(_rn(mid * Fraction(m)))
    bad = [x for x in xs if _markstein64(x, m, inv) != _rn(Fraction(x) / Fraction(m))]
    assert not bad, bad[:5]


def _rn_binary(v: Fraction, p: int, emin: int) -> Fraction:
    """v rounded to nearest-even in a binary format of p significant bits
    and minimum normal exponent emin (no overflow in this use)."""
    if v == 0:
        return v
    a = abs(v)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    quantum = Fraction(2) ** (max(e, emin) - (p - 1))
    n = a / quantum
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return (1 if v > 0 else -1) * fl * quantum


def rn32(v):
    return _rn_binary(v, 24, -126)


def rn16(v):
    return _rn_binary(v, 11, -14)


def test_rounding_helpers_match_numpy():
    rng = random.Random(5)
    for _ in range(2000):
        x = rng.uniform(-65000, 65000) * 2.0 ** rng.randint(-30, 0)
        assert float(rn32(Fraction(x))) == float(np.float32(x))
        assert float(rn16(Fraction(x))) == float(np.float16(x))


def test_binary16_division_by_mass_every_dividend():
    # the binary16 step divides binary16 values by m = RN16(RN16(0.1) + 1)
    # through binary32 (product with RN32(1/m), one fused correction) and
    # rounds once to binary16; it must give RN16 of the exact quotient, as
    # the oracle's binary16 division does
    m = Fraction(float(np.float16(np.float16(0.1) + np.float16(1.0))))
    assert m == Fraction(1126, 1024)
    inv = rn32(1 / m)
    bits = np.arange(0, 0x7C00, dtype=np.uint16)  # every finite non-negative binary16
    bad = []
    for x in bits.view(np.float16).astype(np.float64):
        fx = Fraction(float(x))
        q = rn32(fx * inv)
        r = rn32(fx - q * m)
        q2 = rn32(r * inv + q)
        if rn16(q2) != rn16(fx / m):
            bad.append(float(x))
    assert not bad, bad[:5]  # negative dividends mirror these exactly

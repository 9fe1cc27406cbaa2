"""The binary16 sin/cos table the two-environments-per-lane binary16 kernel
reads (paper_2301_13062_amd/csrc/cp_f16_table.h, evaluated at compile
time): built here with the host compiler from the same header and compared,
entry by entry over every binary16 angle in [0, 1/4], with the C library's
binary64 sin and cos (Python's math module) rounded once to binary16 by
numpy -- the rounding the binary16 step's definition asks for."""
import math
import os
import subprocess

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_every_entry_is_the_rounded_sin_and_cos(tmp_path):
    exe = tmp_path / "f16_table_dump"
    subprocess.run(["g++", "-std=c++17", "-O2",
                    "-I" + os.path.join(ROOT, "paper_2301_13062_amd", "csrc"),
                    os.path.join(ROOT, "tests", "f16_table_dump.cpp"), "-o", str(exe)],
                   check=True, capture_output=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split()
    vals = np.array([int(v, 16) for v in out], dtype=np.uint64)
    n_den = 0x3955 - 0x38F8 + 1
    tab, rec, rec_c = vals[:0x3401], vals[0x3401:0x3401 + n_den], vals[0x3401 + n_den:]
    # bit patterns 0 .. 0x3400 (= 0.25), then 94 divisors, then 65 cosines
    assert len(rec) == n_den and len(rec_c) == 0x3C00 - 0x3BC0 + 1
    x = np.arange(len(tab), dtype=np.uint16).view(np.float16).astype(np.float64)
    assert x[-1] == 0.25 and x[1] == 2.0 ** -24
    sin16 = np.array([np.float16(math.sin(v)) for v in x]).view(np.uint16)
    cos16 = np.array([np.float16(math.cos(v)) for v in x]).view(np.uint16)
    assert np.array_equal(tab & 0xFFFF, sin16.astype(np.uint64))
    assert np.array_equal(tab >> 16, cos16.astype(np.uint64))
    # the divisor reciprocals: the binary32 value nearest to 1/d, decided with
    # exact rationals
    from fractions import Fraction

    def nearest32(r, d):
        got = Fraction(float(np.uint32(r).view(np.float32)))
        e = got.numerator.bit_length() - got.denominator.bit_length()
        if got < Fraction(2) ** e:
            e -= 1  # now 2^e <= got < 2^(e + 1)
        ulp = Fraction(2) ** (e - 23)
        return abs(got - 1 / d) <= ulp / 2

    for k, r in enumerate(rec):
        assert nearest32(r, Fraction(float(np.uint16(0x38F8 + k).view(np.float16)))), k
    # keyed by the cosine: every table cosine is in 0x3BC0 .. 0x3C00, and
    # entry c holds RN32(1 / d(c)), d(c) rounded as the binary16 step rounds
    # it (numpy binary16 rounding of each binary64 operation)
    assert (tab >> 16).min() == 0x3BC0 and (tab >> 16).max() == 0x3C00

    def f16(v):
        return float(np.float16(v))

    mp, four3 = f16(0.1), f16(4.0 / 3.0)
    m = f16(mp + 1.0)
    for k, r in enumerate(rec_c):
        c = float(np.uint16(0x3BC0 + k).view(np.float16))
        d = f16(0.5 * f16(four3 - f16(f16(mp * f16(c * c)) / m)))
        assert nearest32(r, Fraction(d)), k


def test_the_divisors_are_every_one_the_step_can_form():
    # l (4/3 - RN16(RN16(mp c^2) / M)) for every binary16 cosine in [-1, 1],
    # each operation rounded to binary16, is one of the 94 consecutive
    # binary16 values 0x38F8 .. 0x3955 and takes all of them
    h = np.arange(0x10000, dtype=np.uint32).astype(np.uint16).view(np.float16)
    c = h[np.isfinite(h) & (np.abs(h.astype(np.float64)) <= 1)].astype(np.float64)

    def f16(v):
        return np.asarray(v, np.float64).astype(np.float16).astype(np.float64)

    c2 = f16(c * c)
    q = f16(f16(f16(0.1) * c2) / f16(f16(0.1) + 1.0))
    den = np.unique(f16(0.5 * f16(f16(4.0 / 3.0) - q)).astype(np.float16).view(np.uint16))
    assert np.array_equal(den, np.arange(0x38F8, 0x3956, dtype=np.uint16))

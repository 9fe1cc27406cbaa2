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
    tab, rec = vals[:0x3401], vals[0x3401:]
    assert len(rec) == 0x3955 - 0x38F8 + 1  # bit patterns 0 .. 0x3400 (= 0.25), then 94 divisors
    x = np.arange(len(tab), dtype=np.uint16).view(np.float16).astype(np.float64)
    assert x[-1] == 0.25 and x[1] == 2.0 ** -24
    sin16 = np.array([np.float16(math.sin(v)) for v in x]).view(np.uint16)
    cos16 = np.array([np.float16(math.cos(v)) for v in x]).view(np.uint16)
    assert np.array_equal(tab & 0xFFFF, sin16.astype(np.uint64))
    assert np.array_equal(tab >> 16, cos16.astype(np.uint64))
    # the divisor reciprocals: the binary32 value nearest to 1/d, decided with
    # exact rationals
    from fractions import Fraction

    for k, r in enumerate(rec):
        d = Fraction(float(np.uint16(0x38F8 + k).view(np.float16)))
        got = Fraction(float(np.uint32(r).view(np.float32)))
        e = got.numerator.bit_length() - got.denominator.bit_length()
        if got < Fraction(2) ** e:
            e -= 1  # now 2^e <= got < 2^(e + 1)
        ulp = Fraction(2) ** (e - 23)
        assert abs(got - 1 / d) <= ulp / 2, k


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

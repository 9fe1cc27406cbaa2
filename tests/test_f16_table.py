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
    tab = np.array([int(v, 16) for v in out], dtype=np.uint64)
    assert len(tab) == 0x3401  # bit patterns 0 .. 0x3400 (= 0.25)
    x = np.arange(len(tab), dtype=np.uint16).view(np.float16).astype(np.float64)
    assert x[-1] == 0.25 and x[1] == 2.0 ** -24
    sin16 = np.array([np.float16(math.sin(v)) for v in x]).view(np.uint16)
    cos16 = np.array([np.float16(math.cos(v)) for v in x]).view(np.uint16)
    assert np.array_equal(tab & 0xFFFF, sin16.astype(np.uint64))
    assert np.array_equal(tab >> 16, cos16.astype(np.uint64))

"""Build libcpref.so for gfx950: measurement references for the benchmark
(issue rates by vector-instruction class, per-launch floors of graph replay).
Not part of the cart-pole library; bench.py loads it, nothing else does."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = ["ref_valu.hip", "ref_latency.hip"]
OUT_DIR = os.path.join(HERE, "_build")
LIB = os.path.join(OUT_DIR, "libcpref.so")


def flags():
    # the cart-pole library's flags, so that the references compile as the
    # kernels they are read against do
    sys.path.insert(0, ROOT)
    from paper_2301_13062_amd import build as B

    return B.FLAGS


def build(verbose=False) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    tmp = LIB + ".tmp"
    cmd = ["hipcc", *flags(), *[os.path.join(HERE, s) for s in SOURCES], "-o", tmp]
    if verbose:
        print(" ".join(cmd))
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))

"""Build the CPU oracle (test infrastructure only) into oracle/libevox_ref.so,
and the all-core CPU baseline built from it into oracle/libevox_ref_mt.so.

Plain gcc, no fast-math, no floating-point contraction: each float operation
in the oracle is one IEEE rounding and fma appears only where fmaf() is
written.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "evox_ref.c")
OUT = os.path.join(HERE, "libevox_ref.so")


MT_SRC = os.path.join(HERE, "evox_ref_mt.c")
MT_OUT = os.path.join(HERE, "libevox_ref_mt.so")
FLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", "-Wall", "-Wextra"]


def build(verbose: bool = False) -> str:
    """The oracle, and the all-core CPU baseline (the oracle compiled with its
    row loops split over POSIX threads, evox_ref_mt.c)."""
    for src, out, extra in ((SRC, OUT, []), (MT_SRC, MT_OUT, ["-pthread"])):
        cmd = ["gcc"] + FLAGS + extra + ["-o", out + ".tmp", src, "-lm"]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        os.replace(out + ".tmp", out)
    return OUT


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)

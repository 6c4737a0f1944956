"""Build the CPU oracle shared library (test infrastructure only).

`python oracle/build.py` compiles oracle/lamp_oracle.c into
oracle/liblamp_oracle.so with gcc, OpenMP and -ffp-contract=off (every fused
multiply-add in the oracle is an explicit fma call).
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "lamp_oracle.c")
LIB = os.path.join(HERE, "liblamp_oracle.so")


def _has_fma():
    try:
        with open("/proc/cpuinfo") as f:
            return " fma " in f.read()
    except OSError:
        return False


def build(verbose=False):
    flags = ["-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
             "-fno-fast-math", "-Wall", "-Wno-unused-function"]
    if _has_fma():
        # Hardware FMA makes fma()/fmaf() fast; the results are the IEEE fused
        # operation either way.
        flags.append("-mfma")
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc"] + flags + [SRC, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)

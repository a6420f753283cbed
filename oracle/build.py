"""Build the CPU oracle shared library (oracle/libkbo.so) with gcc.

Test infrastructure: the flags keep binary32 arithmetic unfused and IEEE
(no -ffast-math, no -march, -ffp-contract=off).
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libkbo.so")
SOURCES = [os.path.join(HERE, "kbo.c"), os.path.join(HERE, "kbo_rung.c"), os.path.join(HERE, "kbo_derived.c")]
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
          "-Wall", "-Wextra"]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", *CFLAGS, *SOURCES, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

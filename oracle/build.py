"""Build the CPU test oracle (plain C, gcc) into oracle/libsvoracle.so.

Test infrastructure only.  -ffp-contract=off keeps every float operation of
sv_oracle.c a separate IEEE-754 operation rounded to nearest-even; no
-ffast-math, no vectorisation flags.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "sv_oracle.c")
LIB = os.path.join(HERE, "libsvoracle.so")

CFLAGS = ["-std=gnu11", "-O2", "-ffp-contract=off", "-fno-fast-math",
          "-fno-tree-vectorize", "-fPIC", "-shared", "-Wall", "-Wextra"]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", *CFLAGS, SRC, "-o", tmp, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

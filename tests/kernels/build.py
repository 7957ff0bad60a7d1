"""Builds the candidate kernels of the performance-stage tests into a gfx950
code object, tests/kernels/candidates.hsaco (called by __graft_entry__.build)."""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "candidates.hip")
OUT = os.path.join(HERE, "candidates.hsaco")


def build(verbose: bool = False) -> str:
    cmd = ["hipcc", "--genco", "--offload-arch=" + os.environ.get("SV_OFFLOAD_ARCH", "gfx950"), "-O3",
           "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", SRC, "-o", OUT]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("building %s failed:\n%s" % (SRC, res.stderr))
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

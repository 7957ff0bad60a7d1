"""Build libsynthverify.so (gfx950) in-tree with hipcc.

Flags that the numerics depend on:
  -ffp-contract=off                      every a + b * c stays two roundings
  -fno-gpu-flush-denormals-to-zero       fp32 denormals survive synthesis and checks
  -fhip-fp32-correctly-rounded-divide-sqrt  IEEE fp32 division and square root
  no -ffast-math
Packed fp32 instructions are disabled for the device code.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
SOURCES = ["sv_api.hip", "sv_synth.hip", "sv_perturb.hip", "sv_compare.hip", "sv_perf.hip", "sv_files.hip"]
LIB = os.path.join(HERE, "libsynthverify.so")
ARCH = os.environ.get("SV_OFFLOAD_ARCH", "gfx950")

FLAGS = ["-O3", "-std=c++17", "-fPIC", "-shared", "--offload-arch=" + ARCH,
         "-ffp-contract=off", "-fno-gpu-flush-denormals-to-zero",
         "-fhip-fp32-correctly-rounded-divide-sqrt",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function",
         "-I" + os.path.join(ROOT, "include"), "-I" + CSRC]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 feature; that warning is noise
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed (%d):\n%s" % (res.returncode, err))
    if verbose and err.strip():
        print(err, file=sys.stderr)


def build(verbose: bool = False) -> str:
    """Compiles every source to an object (in parallel), then links the library."""
    import tempfile
    from concurrent.futures import ThreadPoolExecutor
    tmp = LIB + ".tmp%d" % os.getpid()
    with tempfile.TemporaryDirectory(prefix="sv_build_") as d:
        objs = [os.path.join(d, os.path.splitext(s)[0] + ".o") for s in SOURCES]
        compile_flags = [f for f in FLAGS if f != "-shared"]
        jobs = [["hipcc", *compile_flags, "-c", os.path.join(CSRC, s), "-o", o] for s, o in zip(SOURCES, objs)]
        with ThreadPoolExecutor(min(len(jobs), os.cpu_count() or 1)) as ex:
            list(ex.map(lambda c: _run(c, verbose), jobs))
        _run(["hipcc", "-shared", "-fPIC", "--offload-arch=" + ARCH, *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))

"""The library's host code built with AddressSanitizer and UndefinedBehaviorSanitizer.

The entry points validate every argument, format their error messages and
keep per-thread state on the host before any HIP call; the CPU tests of the
C ABI (test_abi.py) drive exactly those paths.  This test builds
libsynthverify.so with both sanitizers on its host code only (the gfx950 code
is built as usual: no sanitizer runs on the GPU), lays out a copy of the
package, the header, the oracle and the ABI tests around it, and runs those
tests against it in a process that preloads the sanitizer runtime, stopping at
the first report.
"""
import glob
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PKG = os.path.join(ROOT, "paper_2609_00058_amd")
NOISE = "is not a recognized feature for this target"


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


@pytest.mark.skipif(shutil.which("hipcc") is None or _asan_runtime() is None,
                    reason="hipcc or its AddressSanitizer runtime not available")
def test_abi_tests_pass_on_a_host_sanitized_build():
    sys.path.insert(0, PKG)
    try:
        import build as lib_build
    finally:
        sys.path.pop(0)
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = [f for f in lib_build.FLAGS if f not in ("-shared", "-O3")] + ["-O1", "-g"] + san
    with tempfile.TemporaryDirectory() as tmp:
        # the tree the ABI tests expect: package, header, oracle, tests
        pkg = os.path.join(tmp, "paper_2609_00058_amd")
        os.makedirs(pkg)
        shutil.copy(os.path.join(PKG, "__init__.py"), pkg)
        shutil.copytree(os.path.join(ROOT, "include"), os.path.join(tmp, "include"))
        shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(tmp, "oracle"),
                        ignore=shutil.ignore_patterns("__pycache__"))
        shutil.copytree(HERE, os.path.join(tmp, "tests"), ignore=shutil.ignore_patterns("__pycache__"))
        shutil.copy(os.path.join(ROOT, "pytest.ini"), tmp)

        objs = [os.path.join(tmp, s.replace(".hip", ".o")) for s in lib_build.SOURCES]
        jobs = [["hipcc", *flags, "-c", os.path.join(lib_build.CSRC, s), "-o", o]
                for s, o in zip(lib_build.SOURCES, objs)]

        def run(cmd):
            r = subprocess.run(cmd, capture_output=True, text=True)
            assert r.returncode == 0, "\n".join(l for l in r.stderr.splitlines() if NOISE not in l)[-3000:]

        with ThreadPoolExecutor(min(len(jobs), os.cpu_count() or 1)) as ex:
            list(ex.map(run, jobs))
        run(["hipcc", "-shared", "-fPIC", "--offload-arch=" + lib_build.ARCH, "-Xarch_host", "-fsanitize=address",
             "-Xarch_host", "-fsanitize=undefined", "-shared-libsan", *objs,
             "-o", os.path.join(pkg, "libsynthverify.so")])

        with open(os.path.join(pkg, "libsynthverify.so"), "rb") as f:
            assert b"__asan_init" in f.read()              # the host code is instrumented
        env = dict(os.environ, LD_PRELOAD=_asan_runtime(),
                   ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",   # the interpreter's own allocations stay out
                   UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
        env.pop("PYTHONPATH", None)
        where = subprocess.run([sys.executable, "-c", "import paper_2609_00058_amd as sv; print(sv.LIB_PATH)"],
                               cwd=tmp, env=env, capture_output=True, text=True, timeout=300)
        assert where.returncode == 0 and where.stdout.strip().startswith(tmp), where.stdout + where.stderr
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-m", "not gpu", "tests/test_abi.py"],
                           cwd=tmp, env=env, capture_output=True, text=True, timeout=900)
        out = r.stdout + r.stderr
        assert r.returncode == 0, out[-5000:]
        assert "AddressSanitizer" not in out and "runtime error" not in out, out[-5000:]
        assert " passed" in r.stdout

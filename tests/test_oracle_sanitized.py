"""The CPU oracle built with AddressSanitizer and UndefinedBehaviorSanitizer.

The oracle decides parity, so a stray read past a buffer or an undefined
shift in it would corrupt what every GPU test is compared with.  This test
compiles sv_oracle.c with a driver that calls each of its entry points over
empty, one-element and ragged sizes, window offsets beyond 2^32 and every
element type and distribution (tests/oracle_sanitize_driver.c), with both
sanitizers set to stop at the first report, and runs it.
"""
import os
import shutil
import subprocess
import tempfile

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def _sanitizers_work(cc, tmp):
    src = os.path.join(tmp, "probe.c")
    with open(src, "w") as f:
        f.write("int main(void) { return 0; }\n")
    exe = os.path.join(tmp, "probe")
    r = subprocess.run([cc, "-fsanitize=address,undefined", src, "-o", exe], capture_output=True)
    return r.returncode == 0 and subprocess.run([exe], capture_output=True).returncode == 0


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_runs_clean_under_address_and_undefined_behaviour_sanitizers():
    with tempfile.TemporaryDirectory() as tmp:
        if not _sanitizers_work("gcc", tmp):
            pytest.skip("gcc cannot build sanitized programs here")
        exe = os.path.join(tmp, "driver")
        subprocess.run(["gcc", "-std=gnu11", "-O1", "-g", "-ffp-contract=off", "-fno-fast-math",
                        "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
                        "-I", os.path.join(ROOT, "oracle"),
                        os.path.join(ROOT, "oracle", "sv_oracle.c"), os.path.join(HERE, "oracle_sanitize_driver.c"),
                        "-lm", "-o", exe], check=True, capture_output=True)
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1",
                   UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
        r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
        assert r.returncode == 0, r.stderr[-4000:]
        assert r.stdout.strip().endswith("ok"), r.stdout[-2000:]
        assert "runtime error" not in r.stderr, r.stderr[-4000:]

"""bench.py's command line: one GPU only (a larger --gpus exits with status 2
and says so), step counts checked before any device work, workload names
checked.  CPU only: every case ends before the GPU is touched."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=120, cwd=ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    for n in ("2", "8"):
        r = _bench("--gpus", n)
        assert r.returncode == 2 and "--gpus 1" in r.stderr and r.stdout == ""


def test_bad_step_counts_and_workloads_are_refused():
    for args in (("--steps", "0"), ("--warmup", "-1"), ("--workload", "no_such_workload")):
        r = _bench(*args)
        assert r.returncode == 2 and r.stdout == "", args


def test_workload_names_match_the_workloads_module():
    sys.path.insert(0, ROOT)
    import bench
    import workloads
    assert set(bench.WORKLOAD_NAMES) == set(workloads.WORKLOADS)

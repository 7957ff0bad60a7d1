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


def test_window_reports_merge_into_the_whole_tensor_report(oracle):
    """The all-threads leg of the CPU baseline checks a tensor in windows and
    merges their reports; the merge must give the oracle's report of the whole
    tensor (the fp64 sum within 1e-15 relative: a different summation order)."""
    import numpy as np
    sys.path.insert(0, ROOT)
    import bench
    rng = np.random.default_rng(4)
    n = 100_003
    ref = rng.normal(0, 10, n).astype(np.float32)
    cand = (ref * (1 + rng.normal(0, 1e-6, n))).astype(np.float32)
    cand[[5, 777, 50_000]] = np.float32(np.nan)
    ref[[9, 60_000]] = np.float32(np.inf)
    whole = oracle.compare(ref.view(np.uint32), cand.view(np.uint32), "f32", 1e-6, 0.0, False)
    for parts in (1, 7, 16):
        step = -(-n // parts)
        wins = [(o, min(step, n - o)) for o in range(0, n, step)]
        got = bench.merge_reports([(o, oracle.compare(ref[o:o + m].view(np.uint32), cand[o:o + m].view(np.uint32),
                                                      "f32", 1e-6, 0.0, False)) for o, m in wins])
        for k, v in whole.items():
            if k == "err_sum":
                assert abs(got[k] - v) <= 1e-15 * abs(v)
            else:
                assert got[k] == v, (parts, k)


def test_cpu_baseline_reports_both_legs_and_the_host(oracle):
    sys.path.insert(0, ROOT)
    import bench
    import workloads
    cb = bench.cpu_baseline(workloads.uniform_small(), min_seconds=0.01, max_elems=1 << 14)
    assert cb["kind"] == "oracle" and cb["unit"] == "GB/s" and cb["value"] > 0 and cb["value_1_thread"] > 0
    assert 1 <= cb["cores"] <= 16 and cb["cpu"] and "threads" in cb["sample"]

"""The C-ABI library loads, exports every symbol include/sv.h declares, and
rejects bad arguments with the documented status before any HIP call (no
GPU is needed for any of this)."""
import ctypes
import math
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sv.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(sv_\w+)\s*\(", src, flags=re.M)))


@pytest.fixture(scope="module")
def svlib():
    import paper_2609_00058_amd as sv
    return sv


def test_every_declared_symbol_is_exported(svlib):
    names = declared_functions()
    assert len(names) >= 10
    assert set(names) == set(svlib.SYMBOLS)
    out = subprocess.run(["nm", "-D", "--defined-only", svlib.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(line.split()[-1] for line in out.splitlines() if line.strip())
    for name in names:
        assert name in exported, name
        assert getattr(svlib.lib(), name) is not None


def test_abi_version_and_enums_match_header(svlib):
    L = svlib.lib()
    L.sv_abi_version.restype = ctypes.c_int
    assert L.sv_abi_version() == 1
    src = open(HEADER).read()
    for name, code in [("SV_F32", 0), ("SV_BF16", 1), ("SV_I32", 2), ("SV_UNIFORM", 0), ("SV_NORMAL", 1),
                       ("SV_INT_RANGE", 2), ("SV_SPECIAL", 3), ("SV_OP_FAULT_AT", 6)]:
        assert re.search(r"\b%s = %d\b" % (name, code), src), name
    assert svlib.DTYPE_CODES == {"f32": 0, "bf16": 1, "i32": 2, "f16": 3, "f64": 4, "u8": 5, "i64": 6}
    assert re.search(r"\bSV_PERMUTATION = 4\b", src)
    import oracle as _o
    assert _o.DISTS == svlib.DIST_CODES
    for name, code in [("SV_F16", 3), ("SV_F64", 4), ("SV_U8", 5), ("SV_I64", 6)]:
        assert re.search(r"\b%s = %d\b" % (name, code), src), name
    import oracle
    assert oracle.DTYPES == svlib.DTYPE_CODES
    assert re.search(r"#define SV_MAX_PENDING_CHECKS %d\b" % svlib.SV_MAX_PENDING_CHECKS, src)


def test_struct_layouts_match_the_c_compiler(svlib, tmp_path):
    # sizes and field offsets of every ABI struct, as gcc lays them out from include/sv.h
    mirrors = {"sv_report": svlib.Report, "sv_segment": svlib.Segment,
               "sv_dist_params": svlib.DistParams, "sv_perturb_plan": svlib.PerturbPlan,
               "sv_synth_job": svlib.SynthJob, "sv_launch": svlib.Launch, "sv_timing": svlib.Timing}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "sv.h"', "int main(void) {"]
    for cname, mirror in mirrors.items():
        lines.append('printf("%s %%zu\\n", sizeof(%s));' % (cname, cname))
        for field, _ in mirror._fields_:
            lines.append('printf("%s.%s %%zu\\n", offsetof(%s, %s));' % (cname, field, cname, field))
    lines.append("return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    got = dict(l.split() for l in subprocess.run([str(exe)], capture_output=True, text=True,
                                                   check=True).stdout.splitlines())
    for cname, mirror in mirrors.items():
        assert int(got[cname]) == ctypes.sizeof(mirror), cname
        for field, _ in mirror._fields_:
            assert int(got["%s.%s" % (cname, field)]) == getattr(mirror, field).offset, (cname, field)
    # the numpy form of the report (as_array=True) has the same layout
    assert svlib.REPORT_DTYPE.itemsize == int(got["sv_report"])
    for field, _ in svlib.Report._fields_:
        assert svlib.REPORT_DTYPE.fields[field][1] == int(got["sv_report.%s" % field]), field


def _synth(L, svlib, dtype, dist, n=16, out=0x1000, params=True, **kw):
    p = svlib.dist_params(**kw)
    return L.sv_synth(0, 0, dtype, dist, ctypes.byref(p) if params else None, n, out)


def test_synth_argument_errors_before_any_device_work(svlib):
    L = svlib.lib()
    INV, UNS = svlib.SV_ERR_INVALID_ARG, svlib.SV_ERR_UNSUPPORTED
    assert _synth(L, svlib, 7, 0, a=0.0, b=1.0) == UNS                      # unknown dtype
    assert _synth(L, svlib, 5, 0, a=0.0, b=1.0) == UNS                      # uniform into uint8
    assert _synth(L, svlib, 3, 2, lo=0, hi=3) == UNS                        # int range into fp16
    assert _synth(L, svlib, 5, 2, lo=0, hi=256) == INV                      # beyond uint8
    assert _synth(L, svlib, 6, 2, lo=3, hi=2) == INV
    assert _synth(L, svlib, 4, 0, out=0x1004, a=0.0, b=1.0) == INV          # misaligned fp64
    assert _synth(L, svlib, 0, 9, a=0.0, b=1.0) == UNS                      # unknown dist
    # permutation: integer types only, at most 2^60 values, no more elements than values
    assert _synth(L, svlib, 0, 4, lo=0, hi=9) == UNS                        # fp32
    assert _synth(L, svlib, 2, 4, lo=0, hi=9, n=11) == INV                  # 11 elements of 10 values
    assert _synth(L, svlib, 6, 4, lo=0, hi=2 ** 61, n=4, out=0x1000) == INV
    assert _synth(L, svlib, 5, 4, lo=0, hi=256, n=4) == INV                 # beyond uint8
    assert _synth(L, svlib, 2, 4, lo=5, hi=4, n=0) == INV                   # empty domain
    p = svlib.dist_params(lo=0, hi=99)
    assert L.sv_synth_window(0, 0, 2, 4, ctypes.byref(p), 95, 6, 0x1000) == INV   # past the 100 values
    assert _synth(L, svlib, 0, 2, lo=0, hi=3) == UNS                        # int range into fp32
    assert _synth(L, svlib, 2, 0, a=0.0, b=1.0) == UNS                      # uniform into int32
    assert _synth(L, svlib, 0, 0, params=False) == INV
    assert _synth(L, svlib, 0, 0, out=0, a=0.0, b=1.0) == INV               # NULL with n > 0
    assert _synth(L, svlib, 0, 0, out=0x1002, a=0.0, b=1.0) == INV          # misaligned fp32
    assert _synth(L, svlib, 0, 0, n=1 << 61, a=0.0, b=1.0) == INV           # size overflow
    assert _synth(L, svlib, 0, 0, a=1.0, b=1.0) == INV                      # empty interval
    assert _synth(L, svlib, 0, 0, a=-3e38, b=3e38) == INV                   # span overflows fp32
    assert _synth(L, svlib, 0, 1, mean=0.0, std=-1.0) == INV
    assert _synth(L, svlib, 0, 1, mean=math.nan, std=1.0) == INV
    assert _synth(L, svlib, 0, 3, std=1.0, p_nan=0.6, p_inf=0.6) == INV     # probabilities sum > 1
    assert _synth(L, svlib, 0, 3, std=1.0, p_zero=-0.1) == INV
    assert _synth(L, svlib, 2, 2, lo=5, hi=4) == INV
    assert _synth(L, svlib, 2, 2, lo=0, hi=1 << 31) == INV                  # beyond int32
    assert "int32" in L.sv_last_error().decode()
    assert _synth(L, svlib, 0, 0, n=0, out=0, a=0.0, b=1.0) == svlib.SV_OK  # nothing to do


def test_synth_batched_argument_errors(svlib):
    L = svlib.lib()
    jobs = (svlib.SynthJob * 3)()
    assert L.sv_synth_batched(None, 0) == svlib.SV_OK
    assert L.sv_synth_batched(None, 2) == svlib.SV_ERR_INVALID_ARG
    ok = svlib.dist_params(a=0.0, b=1.0)
    for k in range(3):
        jobs[k] = svlib.SynthJob(1, k, 0, 0, ok, 0, None)          # empty jobs: nothing to launch
    assert L.sv_synth_batched(jobs, 3) == svlib.SV_OK
    jobs[2] = svlib.SynthJob(1, 2, 0, 1, svlib.dist_params(mean=0.0, std=-2.0), 16, 0x1000)
    assert L.sv_synth_batched(jobs, 3) == svlib.SV_ERR_INVALID_ARG
    assert L.sv_last_error().decode().startswith("job 2:")
    jobs[1] = svlib.SynthJob(1, 1, 2, 0, ok, 16, 0x1000)              # uniform into int32
    assert L.sv_synth_batched(jobs, 3) == svlib.SV_ERR_UNSUPPORTED


@pytest.mark.parametrize("entry", ["sv_compare", "sv_compare_noalloc"])
def test_compare_argument_errors_and_empty(svlib, entry):
    L = svlib.lib()
    check = getattr(L, entry)
    INV = svlib.SV_ERR_INVALID_ARG
    rep = svlib.Report()
    assert L.sv_compare(0x1000, 0x2000, 4, 0, 1e-5, 1e-8, 0, None) == INV
    assert L.sv_compare(0, 0x2000, 4, 0, 1e-5, 1e-8, 0, ctypes.byref(rep)) == INV
    assert L.sv_compare(0x1000, 0x2000, 4, 0, -1e-5, 0.0, 0, ctypes.byref(rep)) == INV
    assert L.sv_compare(0x1000, 0x2000, 4, 0, math.inf, 0.0, 0, ctypes.byref(rep)) == INV
    assert L.sv_compare(0x1000, 0x2000, 4, 0, 0.0, math.nan, 0, ctypes.byref(rep)) == INV
    assert L.sv_compare(0x1001, 0x2000, 4, 1, 0.0, 0.0, 0, ctypes.byref(rep)) == INV   # misaligned bf16
    assert L.sv_compare(0x1000, 0x2000, 4, 7, 0.0, 0.0, 0, ctypes.byref(rep)) == svlib.SV_ERR_UNSUPPORTED
    assert "rtol" in L.sv_last_error().decode() or "dtype" in L.sv_last_error().decode()
    assert L.sv_compare(0, 0, 0, 0, 1e-5, 1e-8, 0, ctypes.byref(rep)) == svlib.SV_OK
    assert rep.n == 0 and rep.mismatches == 0 and rep.first_mismatch == -1 and rep.err_sum == 0.0
    # int32 ignores its tolerances, so even invalid values are accepted for it (n = 0 here)
    assert L.sv_compare(0, 0, 0, 2, -1.0, math.nan, 0, ctypes.byref(rep)) == svlib.SV_OK


def test_batched_argument_errors_and_empty(svlib):
    L = svlib.lib()
    segs = (svlib.Segment * 3)()
    reps = (svlib.Report * 3)()
    assert L.sv_compare_batched(None, 0, None) == svlib.SV_OK
    assert L.sv_compare_batched(None, 3, reps) == svlib.SV_ERR_INVALID_ARG
    for k in range(3):
        segs[k] = svlib.Segment(None, None, 0, 0, 1e-5, 1e-8, 0)
    assert L.sv_compare_batched(segs, 3, reps) == svlib.SV_OK
    assert all(reps[k].first_mismatch == -1 for k in range(3))
    segs[1] = svlib.Segment(0x1000, None, 8, 0, 1e-5, 1e-8, 0)
    assert L.sv_compare_batched(segs, 3, reps) == svlib.SV_ERR_INVALID_ARG
    assert "segment 1" in L.sv_last_error().decode()


def test_async_check_argument_errors_without_a_device(svlib):
    L = svlib.lib()
    INV, UNS = svlib.SV_ERR_INVALID_ARG, svlib.SV_ERR_UNSUPPORTED
    t = ctypes.c_uint64(0)
    r = ctypes.c_int32(0)
    reps = (svlib.Report * 2)()
    assert L.sv_compare_submit(0x1000, 0x2000, 4, 0, 1e-5, 1e-8, 0, None) == INV
    assert L.sv_compare_submit(0, 0x2000, 4, 0, 1e-5, 1e-8, 0, ctypes.byref(t)) == INV
    assert L.sv_compare_submit(0x1000, 0x2000, 4, 0, -1.0, 0.0, 0, ctypes.byref(t)) == INV
    assert L.sv_compare_submit(0x1000, 0x2000, 4, 7, 0.0, 0.0, 0, ctypes.byref(t)) == UNS
    segs = (svlib.Segment * 2)()
    segs[0] = svlib.Segment(None, None, 0, 0, 1e-5, 1e-8, 0)
    segs[1] = svlib.Segment(0x1000, None, 8, 0, 1e-5, 1e-8, 0)
    assert L.sv_compare_batched_submit(segs, 2, 0, None) == INV
    assert L.sv_compare_batched_submit(None, 2, 0, ctypes.byref(t)) == INV
    assert L.sv_compare_batched_submit(segs, 2, 5, ctypes.byref(t)) == UNS
    assert L.sv_compare_batched_submit(segs, 2, 0, ctypes.byref(t)) == INV
    assert "segment 1" in L.sv_last_error().decode()
    # tickets that name no device in use, or no device at all
    for bad in (0, 5, (200 << 56) | 3):
        assert L.sv_compare_ready(bad, ctypes.byref(r)) == INV
        assert L.sv_compare_wait(bad, reps, 1) == INV
        assert "ticket" in L.sv_last_error().decode()
    assert L.sv_compare_ready(1 << 56, None) == INV
    # the testing hook refuses sequence numbers that tickets cannot hold
    assert L.sv_testing_set_sequence((1 << 56) - (1 << 32)) == INV
    assert "too large" in L.sv_last_error().decode()


def test_perturb_argument_errors(svlib):
    L = svlib.lib()
    plan = svlib.PerturbPlan(9, 0.5, 0.0, 0, None, 0)
    assert L.sv_perturb(0, 0, 0, ctypes.byref(plan), 4, 0x1000, 0x2000) == svlib.SV_ERR_UNSUPPORTED
    plan = svlib.PerturbPlan(1, 1.5, 0.0, 0, None, 0)
    assert L.sv_perturb(0, 0, 0, ctypes.byref(plan), 4, 0x1000, 0x2000) == svlib.SV_ERR_INVALID_ARG
    plan = svlib.PerturbPlan(1, 0.5, 0.0, 0, None, 0)
    assert L.sv_perturb(0, 0, 2, ctypes.byref(plan), 4, 0x1000, 0x2000) == svlib.SV_ERR_UNSUPPORTED
    idx = (ctypes.c_uint64 * 2)(1, 4)
    plan = svlib.PerturbPlan(5, 0.0, 0.0, 0, idx, 2)
    assert L.sv_perturb(0, 0, 0, ctypes.byref(plan), 4, 0x1000, 0x2000) == svlib.SV_ERR_INVALID_ARG
    assert "out of range" in L.sv_last_error().decode()
    assert L.sv_perturb(0, 0, 0, None, 4, 0x1000, 0x2000) == svlib.SV_ERR_INVALID_ARG


def test_profile_read_with_nothing_recorded(svlib):
    c, ms = svlib.profile_read("synth")
    assert c == 0 and ms == 0.0


def test_eval_transform_argument_errors(svlib):
    L = svlib._lib
    assert L.sv_eval_transform(6, 0x1000, 4, 0x2000) == svlib.SV_ERR_UNSUPPORTED
    assert L.sv_eval_transform(-1, 0x1000, 4, 0x2000) == svlib.SV_ERR_UNSUPPORTED
    assert L.sv_eval_transform(0, None, 4, 0x2000) == svlib.SV_ERR_INVALID_ARG
    assert L.sv_eval_transform(0, 0x1002, 4, 0x2000) == svlib.SV_ERR_INVALID_ARG   # misaligned
    assert L.sv_eval_transform(1, None, 0, None) == svlib.SV_OK


def test_kernel_harness_argument_errors_before_any_device_work(svlib):
    L = svlib.lib()
    INV = svlib.SV_ERR_INVALID_ARG
    h = ctypes.c_void_p()
    assert L.sv_kernel_load(None, 100, b"k", ctypes.byref(h)) == INV
    assert L.sv_kernel_load(b"\x7fELF" + b"\0" * 60, 0, b"k", ctypes.byref(h)) == INV
    assert L.sv_kernel_load(b"\x7fELF" + b"\0" * 60, 64, None, ctypes.byref(h)) == INV
    assert L.sv_kernel_load(b"not a code object at all", 24, b"k", ctypes.byref(h)) == INV
    assert "code object" in L.sv_last_error().decode()
    l = svlib.Launch((ctypes.c_uint32 * 3)(1, 1, 1), (ctypes.c_uint32 * 3)(64, 1, 1), 0, 0, None, 0)
    t = svlib.Timing()
    assert L.sv_kernel_launch(None, ctypes.byref(l)) == INV
    assert L.sv_kernel_time(None, ctypes.byref(l), 0, 10, 0, None, ctypes.byref(t)) == INV
    assert L.sv_kernel_free(None) == svlib.SV_OK


def test_reward_matches_the_oracle_on_every_case(svlib, oracle):
    L = svlib.lib()
    for c in (0, 1):
        for v in (0, 1):
            for p in (0.0, 0.5, 2.0, 1e6, math.inf):
                want = oracle.reward(c, v, p)
                got = L.sv_reward(c, v, p)
                assert got == want, (c, v, p, got, want)
    assert math.isnan(L.sv_reward(1, 1, -1.0)) and math.isnan(L.sv_reward(1, 1, math.nan))
    assert L.sv_reward(0, 1, math.nan) == -1.0 and L.sv_reward(1, 0, math.nan) == 0.0
    assert svlib.reward(True, True, 4.0) == 4.0


def test_wall_clock_attribute_value_used_by_the_gpu_tests(tmp_path):
    src = tmp_path / "wc.cpp"
    src.write_text('#include <hip/hip_runtime_api.h>\n#include <cstdio>\n'
                   'int main() { printf("%d", (int)hipDeviceAttributeWallClockRate); return 0; }\n')
    exe = tmp_path / "wc"
    subprocess.run(["g++", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", str(src), "-o", str(exe)], check=True)
    import test_gpu_perf
    assert int(subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout) == \
        test_gpu_perf.WALL_CLOCK_RATE_ATTR


def test_file_entry_points_reject_bad_arguments_without_a_device(svlib, tmp_path):
    L = svlib.lib()
    p = svlib.dist_params(a=-1.0, b=1.0)
    assert L.sv_synth_file(None, 0, 0, 0, 0, ctypes.byref(p), 10) == svlib.SV_ERR_INVALID_ARG
    assert L.sv_synth_file(str(tmp_path / "x").encode(), 0, 0, 2, 0, ctypes.byref(p), 10) == \
        svlib.SV_ERR_UNSUPPORTED                      # int32 from a uniform distribution
    assert not (tmp_path / "x").exists()              # nothing created for invalid arguments
    r = svlib.Report()
    assert L.sv_compare_file(b"/nonexistent/ref", b"/nonexistent/cand", 4, 0, 0.0, 0.0, 0,
                             ctypes.byref(r)) == svlib.SV_ERR_IO
    assert "cannot open" in L.sv_last_error().decode()
    a, b = tmp_path / "a.bin", tmp_path / "b.bin"
    a.write_bytes(b"\0" * 16)
    b.write_bytes(b"\0" * 12)
    assert L.sv_compare_file(str(a).encode(), str(b).encode(), 4, 0, 0.0, 0.0, 0, ctypes.byref(r)) == \
        svlib.SV_ERR_INVALID_ARG                      # 12 bytes are not 4 fp32 values
    assert "holds 12 bytes" in L.sv_last_error().decode()
    assert L.sv_compare_file(str(a).encode(), str(a).encode(), 4, 0, -1.0, 0.0, 0, ctypes.byref(r)) == \
        svlib.SV_ERR_INVALID_ARG                      # tolerance checked as in sv_compare
    assert L.sv_compare_file(str(a).encode(), str(a).encode(), 0, 0, 0.0, 0.0, 0, ctypes.byref(r)) == \
        svlib.SV_ERR_INVALID_ARG                      # 16 bytes are not 0 values
    q = svlib.dist_params(a=-1.0, b=1.0)
    assert L.sv_synth_window(0, 0, 0, 0, ctypes.byref(q), 1 << 60, 1, 0x1000) == svlib.SV_ERR_INVALID_ARG


def test_one_hip_runtime_per_process_with_torch():
    """The package loads torch before the library, so the library binds to
    the HIP runtime torch ships and the process maps one copy of it (two
    copies left the library without a device)."""
    code = ("import paper_2609_00058_amd\n"
            "paths = sorted({l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l})\n"
            "print('\\n'.join(paths))\n")
    r = subprocess.run([__import__("sys").executable, "-c", code], cwd=ROOT, capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    paths = r.stdout.split()
    assert len(paths) == 1, paths
    import torch
    assert os.path.dirname(paths[0]) == os.path.join(os.path.dirname(torch.__file__), "lib"), paths

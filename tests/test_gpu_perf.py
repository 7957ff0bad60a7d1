"""GPU tests of the performance stage (Eq. 3) and the reward (Eq. 4): the
harness times a kernel of known duration correctly, its statistics are those
of the per-run times, and the whole fail-fast sequence (functional check,
then profiling, then reward) ranks a correct and a faulty candidate."""
import ctypes
import os
import struct

import numpy as np
import pytest
import torch

import paper_2609_00058_amd as sv

pytestmark = pytest.mark.gpu

HSACO = os.path.join(os.path.dirname(os.path.abspath(__file__)), "kernels", "candidates.hsaco")
WALL_CLOCK_RATE_ATTR = 10017   # hipDeviceAttributeWallClockRate (kHz); checked against the header in test_abi


@pytest.fixture(scope="module")
def code():
    if not os.path.exists(HSACO):
        pytest.fail("tests/kernels/candidates.hsaco is not built (run __graft_entry__.build())")
    with open(HSACO, "rb") as f:
        return f.read()


def wall_clock_mhz():
    rate = ctypes.c_int()
    hip = ctypes.CDLL("libamdhip64.so.7")   # by its soname: the runtime torch has loaded, not a second copy
    assert hip.hipDeviceGetAttribute(ctypes.byref(rate), WALL_CLOCK_RATE_ATTR, 0) == 0
    return rate.value / 1e3


def test_known_duration_is_measured(code):
    torch.cuda.set_device(0)
    k = sv.kernel_load(code, "sv_test_spin")
    mhz = wall_clock_mhz()
    assert 1 <= mhz <= 1000, mhz
    for us in (50.0, 400.0, 2000.0):
        print("spin", us, "us", flush=True)
        t = k.time((1,), (64,), struct.pack("<Q", int(us * mhz)), warmup=2, reps=15, per_rep=True)
        assert t["reps"] == 15 and len(t["rep_ms"]) == 15
        ms = np.array(t["rep_ms"], dtype=np.float64)
        assert t["mean_ms"] == pytest.approx(ms.mean(), rel=1e-12)
        assert t["min_ms"] == ms.min() and t["max_ms"] == ms.max()
        assert t["median_ms"] == pytest.approx(float(np.median(ms)), rel=1e-12)
        assert t["perf"] == 1.0 / t["mean_ms"]
        # the spin lasts at least `us`; events and dispatch add a few microseconds
        assert us * 1e-3 <= t["min_ms"] and t["mean_ms"] <= us * 1e-3 * 1.02 + 0.02, t
    k.free()


def test_empty_kernel_and_flush(code):
    k = sv.kernel_load(code, "sv_test_empty")
    t = k.time((1,), (64,), warmup=1, reps=50)
    assert 0 < t["min_ms"] <= t["median_ms"] <= t["max_ms"] < 1.0, t
    print("empty kernel", t, flush=True)
    t2 = k.time((1,), (64,), warmup=1, reps=5, flush_bytes=256 << 20)
    assert 0 < t2["mean_ms"] < 1.0, t2


def _axpy_args(z, x, y, a, n):
    return struct.pack("<QQQfxxxxQ", z.data_ptr(), x.data_ptr(), y.data_ptr(), a, n)


def test_fail_fast_sequence_ranks_candidates(code):
    n = (1 << 22) + 17
    g = torch.Generator().manual_seed(5)
    x = torch.randn(n, generator=g).cuda()
    y = torch.randn(n, generator=g).cuda()
    a = 1.7
    ref = (torch.tensor(a, dtype=torch.float32) * x.cpu() + y.cpu()).cuda()   # two roundings, as the kernel
    grid, block = ((n + 255) // 256,), (256,)
    results = {}
    for name in ("sv_test_axpy", "sv_test_axpy_tail_bug"):
        print("candidate", name, flush=True)
        k = sv.kernel_load(code, name)
        z = torch.zeros(n, device="cuda")
        k.launch(grid, block, _axpy_args(z, x, y, a, n))
        rep = sv.compare(ref, z, 0.0, 0.0)
        valid = rep["mismatches"] == 0
        perf = k.time(grid, block, _axpy_args(z, x, y, a, n), reps=10)["perf"] if valid else 0.0
        results[name] = (rep, valid, perf, sv.reward(True, valid, perf))
        k.free()
    rep, valid, perf, r = results["sv_test_axpy"]
    assert valid and rep["max_abs_err"] == 0.0 and perf > 0 and r == perf
    rep, valid, perf, r = results["sv_test_axpy_tail_bug"]
    assert not valid and rep["mismatches"] == 1 and rep["first_mismatch"] == n - 1 and r == 0.0
    assert sv.reward(False, False, 0.0) == -1.0


def test_load_errors_from_the_runtime(code):
    with pytest.raises(sv.SVError) as e:
        sv.kernel_load(code, "no_such_kernel")
    assert e.value.code == sv.SV_ERR_HIP
    torch.empty(16, device="cuda").fill_(1.0)     # the library's failure does not leak into torch
    torch.cuda.synchronize()
    k = sv.kernel_load(code, "sv_test_empty")
    with pytest.raises(sv.SVError) as e:
        k.time((1,), (2048,))
    assert e.value.code == sv.SV_ERR_INVALID_ARG
    with pytest.raises(sv.SVError) as e:
        k.time((0,), (64,))
    assert e.value.code == sv.SV_ERR_INVALID_ARG
    k.free()

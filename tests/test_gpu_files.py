"""GPU parity of window synthesis and of the file entry points: windows are
slices of the whole tensor; files hold exactly the synthesized bits; file
checks report what the oracle reports for the same data, read with the
declared element type."""
import numpy as np
import pytest
import torch

import paper_2609_00058_amd as sv
from gpu_run import bits, empty, same_report

pytestmark = pytest.mark.gpu

SPECIAL = dict(mean=0.0, std=1e3, p_nan=0.01, p_inf=0.005, p_denorm=0.01, p_zero=0.01)
WINDOW_CASES = [("uniform", "f32", dict(a=-1.0, b=1.0)), ("normal", "bf16", dict(mean=5.0, std=10.0)),
                ("int_range", "i32", dict(lo=-1000, hi=1000)), ("special", "f32", SPECIAL),
                ("normal", "f32", dict(mean=0.0, std=1.0)), ("uniform", "bf16", dict(a=-4.0, b=4.0))]


@pytest.mark.parametrize("dist,dtype,params", WINDOW_CASES)
def test_window_is_the_slice_of_the_tensor(oracle, dist, dtype, params):
    full = empty(300_000, dtype)
    sv.synth(full, 7, 3, dist, **params)
    fb = bits(full)
    for off, n in [(0, 1), (4, 1000), (5, 777), (1, 3), (8, 4097), (131_071, 100_000), (131_072, 5000),
                   (299_990, 10)]:
        print("window", dist, dtype, off, n, flush=True)
        big = empty(n + 8, dtype)
        for shift in (0, 1):                        # 16-byte aligned and not
            w = big[shift:shift + n]
            sv.synth_window(w, 7, 3, dist, off, **params)
            assert np.array_equal(bits(w), fb[off:off + n])
        want = oracle.synth(7, 3, dtype, dist, oracle.dist_params(**params), n, off)
        assert np.array_equal(fb[off:off + n], want)
    far = empty(1000, dtype)                         # far from the start: against the oracle alone
    sv.synth_window(far, 7, 3, dist, (1 << 40) + 12, **params)
    assert np.array_equal(bits(far), oracle.synth(7, 3, dtype, dist, oracle.dist_params(**params), 1000,
                                                  (1 << 40) + 12))


@pytest.mark.parametrize("dist,dtype,params,n", [
    ("normal", "f32", dict(mean=5.0, std=10.0), 3 * (1 << 24) + 5),   # three 64 MiB chunks and a tail
    ("uniform", "bf16", dict(a=-4.0, b=4.0), (1 << 25) + 3),
    ("int_range", "i32", dict(lo=-(1 << 20), hi=1 << 20), 1000),
])
def test_synth_file_holds_the_synthesized_bits(oracle, tmp_path, dist, dtype, params, n):
    path = tmp_path / ("%s_%s.bin" % (dist, dtype))
    print("synth file", dist, dtype, n, flush=True)
    sv.synth_file(str(path), n, 11, 2, dtype, dist, **params)
    got = np.fromfile(path, dtype=np.uint16 if dtype == "bf16" else np.uint32)
    assert got.size == n
    want = oracle.synth(11, 2, dtype, dist, oracle.dist_params(**params), n)
    assert np.array_equal(got, want)


def _write(path, arr):
    np.ascontiguousarray(arr).tofile(path)
    return str(path)


def test_compare_file_matches_the_oracle(oracle, tmp_path):
    rng = np.random.default_rng(9)
    for dtype, n in [("f32", (1 << 24) + 17), ("bf16", 1000), ("i32", (1 << 24) + 3), ("f32", 1)]:
        print("compare file", dtype, n, flush=True)
        if dtype == "i32":
            ref = rng.integers(0, 100, n).astype(np.int32)
            cand = ref.copy()
            cand[[0, n // 2, n - 1]] += 1              # tiny ints: as fp32 bits these are denormals
            ref, cand = ref.view(np.uint32), cand.view(np.uint32)
        else:
            ref = rng.normal(5.0, 10.0, n).astype(np.float32)
            cand = ref.copy()
            k = rng.random(n) < 0.01
            cand[k] = cand[k] * np.float32(1.0 + 1e-3)
            cand[n // 3] = np.float32("nan")
            if dtype == "bf16":
                to16 = lambda x: torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
                ref, cand = to16(ref), to16(cand)
            else:
                ref, cand = ref.view(np.uint32), cand.view(np.uint32)
        rp, cp = _write(tmp_path / "r.bin", ref), _write(tmp_path / "c.bin", cand)
        rtol, atol = (1e-5, 1e-6) if dtype != "bf16" else (1e-2, 1e-2)
        got = sv.compare_file(rp, cp, n, dtype, rtol, atol, False)
        want = oracle.compare(ref, cand, dtype, rtol, atol, False)
        same_report(got, want)
        if dtype == "i32":
            assert got["mismatches"] == 3 and got["first_mismatch"] == 0
            # the same bits read as fp32 would pass at this atol: the declared type decides
            assert oracle.compare(ref, cand, "f32", rtol, atol, False)["mismatches"] == 0


def test_compare_file_errors(tmp_path):
    a = _write(tmp_path / "a.bin", np.zeros(10, np.float32))
    with pytest.raises(sv.SVError) as e:
        sv.compare_file(a, str(tmp_path / "missing.bin"), 10, "f32", 0.0, 0.0)
    assert e.value.code == sv.SV_ERR_IO
    with pytest.raises(sv.SVError) as e:
        sv.compare_file(a, a, 11, "f32", 0.0, 0.0)
    assert e.value.code == sv.SV_ERR_INVALID_ARG
    assert sv.compare_file(a, a, 10, "f32", 0.0, 0.0)["mismatches"] == 0
    with pytest.raises(sv.SVError) as e:
        sv.synth_file(str(tmp_path / "no_dir" / "x.bin"), 10, 0, 0, "f32", "uniform", a=-1.0, b=1.0)
    assert e.value.code == sv.SV_ERR_IO

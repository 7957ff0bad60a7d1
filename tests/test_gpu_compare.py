"""GPU parity of sv_compare / sv_compare_batched against the CPU oracle.

Counts, indices and maxima must match bit for bit; the fp64 error sum within
1e-12 relative (exactly 0 when every difference is 0).  Inputs: a grid of
special values, random data with specials at sizes spanning several tiles
and ragged tails, unaligned and differently aligned views, empty tensors,
ragged batches with zero-length and aliased segments, and a tensor longer
than 2^32 elements.
"""
import math

import numpy as np
import pytest
import torch

import paper_2609_00058_amd as sv
from gpu_run import bits, empty, same_report

pytestmark = pytest.mark.gpu

GRID = [0x00000000, 0x80000000, 0x00000001, 0x80000001, 0x00800000, 0x80800000,
        0x3F800000, 0xBF800000, 0x3F800001, 0x3F7FFFFF, 0x7F7FFFFF, 0xFF7FFFFF,
        0x7F800000, 0xFF800000, 0x7FC00000, 0x7FC00001, 0xFFC12345, 0x7F800001,
        0x3A83126F, 0x00400000]
TOLS = [(0.0, 0.0), (1e-5, 1e-8), (1e-2, 1e-2), (0.5, 0.0), (0.0, 2.0 ** -149), (1e-7, 0.0),
        (1.0, 1e-45), (2.0 ** -23, 0.0)]


def dev(bits_np, dtype):
    t = {"f32": torch.int32, "i32": torch.int32, "bf16": torch.int16}[dtype]
    a = torch.from_numpy(np.ascontiguousarray(bits_np).view(np.int16 if dtype == "bf16" else np.int32))
    out = a.to("cuda")
    return out.view({"f32": torch.float32, "i32": torch.int32, "bf16": torch.bfloat16}[dtype])


def random_pair(rng, n, dtype, special_frac=0.05):
    if dtype == "i32":
        ref = rng.integers(-1000, 1000, n).astype(np.int32)
        cand = ref.copy()
        k = rng.random(n) < 0.01
        cand[k] += rng.integers(-3, 4, k.sum()).astype(np.int32)
        return ref.view(np.uint32), cand.view(np.uint32)
    ref = rng.normal(5.0, 10.0, n).astype(np.float32)
    noise = rng.normal(0, 1, n) * np.abs(ref) * 10.0 ** rng.uniform(-9, -2, n)
    cand = (ref.astype(np.float64) + noise).astype(np.float32)
    same = rng.random(n) < 0.2
    cand[same] = ref[same]
    sp = np.array([0x7FC00000, 0xFFC00001, 0x7F800000, 0xFF800000, 0, 0x80000000, 1, 0x80000005],
                  np.uint32).view(np.float32)
    for arr in (ref, cand):
        k = rng.random(n) < special_frac
        arr[k] = rng.choice(sp, k.sum())
    if dtype == "bf16":
        import torch as T
        cvt = lambda x: T.from_numpy(x).to(T.bfloat16).view(T.int16).numpy().view(np.uint16)
        return cvt(ref), cvt(cand)
    return ref.view(np.uint32), cand.view(np.uint32)


def test_special_value_grid_every_pair(oracle):
    # every (candidate, reference) pair of the grid as its own segment of one batch
    a = np.repeat(np.array(GRID, np.uint32), len(GRID))
    y = np.tile(np.array(GRID, np.uint32), len(GRID))
    A, Y = dev(a, "f32"), dev(y, "f32")
    for rtol, atol in TOLS:
        for eqn in (False, True):
            print("grid", rtol, atol, eqn, flush=True)
            segs = [(Y[k:k + 1], A[k:k + 1], rtol, atol, eqn) for k in range(a.size)]
            got = sv.compare_batched(segs)
            for k in range(a.size):
                want = oracle.compare(y[k:k + 1], a[k:k + 1], "f32", rtol, atol, eqn)
                same_report(got[k], want)
            same_report(sv.compare(Y, A, rtol, atol, eqn), oracle.compare(y, a, "f32", rtol, atol, eqn))


@pytest.mark.parametrize("dtype", ["f32", "bf16", "i32"])
def test_random_pairs_all_sizes(oracle, dtype):
    rng = np.random.default_rng(17)
    for n in [1, 5, 63, 64, 65, 1000, 4099, 200003, (1 << 22) + 5]:
        ref, cand = random_pair(rng, n, dtype)
        R, C = dev(ref, dtype), dev(cand, dtype)
        for rtol, atol, eqn in [(1e-5, 1e-8, False), (1e-3, 1e-6, True), (0.0, 0.0, True)]:
            print("random", dtype, n, rtol, atol, eqn, flush=True)
            same_report(sv.compare(R, C, rtol, atol, eqn), oracle.compare(ref, cand, dtype, rtol, atol, eqn))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_unaligned_and_differently_aligned_views(oracle, dtype):
    rng = np.random.default_rng(3)
    n = 70001
    ref, cand = random_pair(rng, n + 16, dtype)
    R, C = dev(ref, dtype), dev(cand, dtype)
    for ro, co in [(1, 1), (1, 2), (0, 3), (5, 0), (8, 8)]:
        print("views", dtype, ro, co, flush=True)
        got = sv.compare(R[ro:ro + n], C[co:co + n], 1e-4, 1e-7, True)
        want = oracle.compare(ref[ro:ro + n], cand[co:co + n], dtype, 1e-4, 1e-7, True)
        same_report(got, want)


def test_empty_and_determinism(oracle):
    e = empty(0, "f32")
    assert sv.compare(e, e, 1e-5, 1e-8) == oracle.compare(np.empty(0, np.uint32), np.empty(0, np.uint32),
                                                           "f32", 1e-5, 1e-8, False)
    rng = np.random.default_rng(8)
    ref, cand = random_pair(rng, 3_000_017, "f32")
    R, C = dev(ref, "f32"), dev(cand, "f32")
    r1 = sv.compare(R, C, 1e-5, 1e-8, False)
    r2 = sv.compare(R, C, 1e-5, 1e-8, False)
    assert r1 == r2
    assert sv.compare_batched([(R, C, 1e-5, 1e-8, False)])[0] == r1


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_single_equals_batched_across_grid_sizes(oracle, dtype):
    # a single tensor is reported by its only workgroup (small), by the last
    # workgroup to finish (up to one wave of workgroups) or by the finalize
    # kernel (larger); a one-segment batch always by the finalize kernel: the
    # reports must be bit-identical, and match the oracle
    rng = np.random.default_rng(9)
    per = 4 if dtype == "f32" else 8
    for units in (1, 4095, 4096, 4097, 16384, 32767, 32768, 32769, 40000, 300000):
        n = units * per - (1 if units > 1 else 0)
        print("single vs batched", dtype, n, flush=True)
        ref, cand = random_pair(rng, n, dtype)
        R, C = dev(ref, dtype), dev(cand, dtype)
        single = sv.compare(R, C, 1e-5, 1e-8, True)
        assert sv.compare_batched([(R, C, 1e-5, 1e-8, True)])[0] == single
        assert sv.compare_submit(R, C, 1e-5, 1e-8, True).wait() == single
        same_report(single, oracle.compare(ref, cand, dtype, 1e-5, 1e-8, True))


def test_bad_arguments_raise():
    x = empty(8, "f32")
    for rtol, atol in [(-1.0, 0.0), (0.0, math.nan), (math.inf, 0.0)]:
        with pytest.raises(sv.SVError) as e:
            sv.compare(x, x, rtol, atol)
        assert e.value.code == sv.SV_ERR_INVALID_ARG


def test_batched_mixed_ragged_aliased(oracle):
    rng = np.random.default_rng(21)
    sizes = [0, 1, 7, 8, 9, 255, 4096, 0, 65537, 1_000_003, 3, 0, 123457]
    segs, want = [], []
    keep = []
    for k, n in enumerate(sizes):
        dtype = ["f32", "bf16", "i32"][k % 3]
        ref, cand = random_pair(rng, n + 3, dtype)
        off = k % 3
        R, C = dev(ref, dtype), dev(cand, dtype)
        keep += [R, C]
        rtol, atol, eqn = [(1e-5, 1e-8, False), (1e-2, 1e-2, True), (1e-3, 0.0, False)][k % 3]
        segs.append((R[off:off + n], C[off:off + n], rtol, atol, eqn))
        want.append(oracle.compare(ref[off:off + n], cand[off:off + n], dtype, rtol, atol, eqn))
        if k % 4 == 0:     # alias: the same pair again, and a pair checked against itself
            segs.append((R[off:off + n], C[off:off + n], rtol, atol, eqn))
            want.append(want[-1])
            segs.append((R[off:off + n], R[off:off + n], rtol, atol, eqn))
            want.append(oracle.compare(ref[off:off + n], ref[off:off + n], dtype, rtol, atol, eqn))
    print("batched mixed", len(segs), flush=True)
    got = sv.compare_batched(segs)
    for g, w in zip(got, want):
        same_report(g, w)
    many = [(s[0][:5], s[1][:5], s[2], s[3], s[4]) for s in segs if s[0].numel() >= 5] * 60
    print("batched many", len(many), flush=True)
    got = sv.compare_batched(many)
    for g, s in zip(got, many):
        same_report(g, sv.compare(*s))
    e = empty(0, "f32")
    assert all(r["first_mismatch"] == -1 and r["n"] == 0 for r in sv.compare_batched([(e, e, 0.0, 0.0, False)] * 3))


def test_indices_beyond_2_pow_32():
    # 2^32 + 17 bf16 elements (8 GiB per operand): one planted fault near the end
    n = (1 << 32) + 17
    print("2^32 + 17 bf16", flush=True)
    ref = empty(n, "bf16")
    sv.synth(ref, 0, 0, "uniform", a=-4.0, b=4.0)
    cand = torch.empty_like(ref)
    sv.perturb(ref, cand, 0, 0, "copy")
    j = (1 << 32) + 9
    sv.perturb(ref, cand, 0, 0, "fault_at", idx=[j])
    rep = sv.compare(ref, cand, 1e-2, 1e-2)
    y = float(ref[j].float())
    a = float(cand[j].float())
    assert rep["n"] == n and rep["mismatches"] == 1 and rep["first_mismatch"] == j
    assert rep["max_abs_err"] == abs(a - y) and rep["err_sum"] == abs(a - y)
    del ref, cand
    torch.cuda.empty_cache()


def _stop_expect(full):
    if full["mismatches"] == 0:
        return full
    out = {k: (0 if isinstance(v, int) else 0.0) for k, v in full.items()}
    out.update(n=full["n"], mismatches=1, first_mismatch=full["first_mismatch"])
    return out


def test_batched_stop_at_first(oracle):
    # G candidates x outputs: clean, wrong from the start, wrong at the very end, one fault in the middle,
    # a NaN against a number, 1 % wrong; the early exit must keep the first index exact
    rng = np.random.default_rng(33)
    segs, want, keep = [], [], []
    for k, n in enumerate([1, 7, 1000, 65537, (1 << 20) + 3, 1 << 22, (1 << 22) + 5, 12345]):
        dtype = ["f32", "bf16", "i32"][k % 3]
        ref, cand = random_pair(rng, n, dtype, special_frac=0.0)
        if dtype == "i32":
            ref_vals = ref.view(np.int32)
        tol = (1e-5, 1e-8, False) if dtype != "bf16" else (1e-2, 1e-2, False)
        R = dev(ref, dtype)
        keep.append(R)
        variants = [ref.copy()]                                  # passes
        bad = ref.copy()
        bad_pos = [0, n - 1, n // 2]
        for pos in bad_pos:                                      # a wrong value at pos
            c = ref.copy()
            if dtype == "i32":
                c.view(np.int32)[pos] += 1
            elif dtype == "bf16":
                c[pos] = 0x7FC0                                  # NaN against a number
            else:
                c[pos] = np.float32(c.view(np.float32)[pos] * 2 + 1).view(np.uint32)
            variants.append(c)
        if n >= 100:
            c = ref.copy()
            idx = rng.choice(n, n // 100, replace=False)
            c[idx] = ref[(idx + 1) % n] if dtype != "i32" else (ref.view(np.int32)[idx] + 7).view(np.uint32)
            variants.append(c)
        for c in variants:
            C = dev(c, dtype)
            keep.append(C)
            segs.append((R, C, *tol))
            want.append(oracle.compare(ref, c, dtype, *tol))
    print("stop-at-first batch", len(segs), flush=True)
    for rep in range(2):                                         # the first call's posted mismatches do not stop the second
        got = sv.compare_batched(segs, stop_at_first=True)
        for g, w in zip(got, want):
            same_report(g, _stop_expect(w))
    got = sv.compare_batched(segs)                               # and the full check is unaffected
    for g, w in zip(got, want):
        same_report(g, w)
    with pytest.raises(sv.SVError) as e:
        arr = (sv.Segment * 1)()
        reps = (sv.Report * 1)()
        sv._check(sv.lib().sv_compare_batched_mode(arr, 1, 2, reps))
    assert e.value.code == sv.SV_ERR_UNSUPPORTED


TILE = 512 * 2          # units per workgroup iteration of a stop-at-first check (threads x units in flight)


def test_stop_at_first_shared_between_workgroups(oracle):
    # In stop-at-first mode a segment's workgroups sweep it together and post the
    # first mismatch they find for the others.  Faults at tile edges, several per
    # segment (a later one may be posted first), segments of one and of thousands
    # of workgroups, unaligned operands (guarded loads only), empty segments
    # between; then the same segments without faults, which must not be stopped by
    # what the first launch posted.
    rng = np.random.default_rng(35)
    E = TILE * 4                                                 # fp32 elements per tile
    cases = [((1 << 24) + 37, [3 * E + 5, 9 * E - 1, 2000 * E]),    # thousands of workgroups
             ((1 << 24) + 37, [(1 << 24) + 36]),                   # the last element
             ((1 << 24) + 37, [0, 12345678]),
             ((1 << 22) + 3, [E - 1, E]),                          # both sides of a tile edge
             ((1 << 22) + 3, [377 * E + 1000, 50 * E + 17, 500 * E + 2, 100 * E]),
             (0, []),
             (5 * E + 3, [4 * E + 1]),                             # one workgroup
             (70_001, [69_999]), (70_001, [40_000, 20_001])]       # unaligned below
    rows, segs, want, keep = [], [], [], []
    for k, (n, faults) in enumerate(cases):
        unaligned = n == 70_001
        ref = rng.normal(0.0, 1.0, n + 1).astype(np.float32).view(np.uint32)
        cand = ref.copy()
        for f in faults:
            cand[f + 1 if unaligned else f] ^= 0x00400000            # far outside rtol
        near = ref ^ np.uint32(1)                                # 1 ulp off everywhere: passes, err_sum > 0
        R, C, N = dev(ref, "f32"), dev(cand, "f32"), dev(near, "f32")
        keep += [R, C, N]
        if unaligned:                                            # views 4 bytes into the storage
            R, C, N, r, c, m = R[1:], C[1:], N[1:], ref[1:], cand[1:], near[1:]
        else:
            R, C, N, r, c, m = R[:n], C[:n], N[:n], ref[:n], cand[:n], near[:n]
        segs.append((R, C, 1e-6, 0.0, False))
        rows.append((r, m, (R, N, 1e-6, 0.0, False)))
        w = oracle.compare(r, c, "f32", 1e-6, 0.0, False)
        assert w["mismatches"] == len(faults) and (not faults or w["first_mismatch"] == min(faults))
        want.append(w)
    print("stop-at-first shared", len(segs), flush=True)
    for rep in range(3):
        got = sv.compare_batched(segs, stop_at_first=True)
        for g, w in zip(got, want):
            same_report(g, _stop_expect(w))
        clean = sv.compare_batched([row[2] for row in rows], stop_at_first=True)
        for g, (r, m, _) in zip(clean, rows):
            w = oracle.compare(r, m, "f32", 1e-6, 0.0, False)
            assert w["mismatches"] == 0 and (w["err_sum"] > 0 or r.size == 0)
            same_report(g, w)
    # many small segments, one failing in four, empty ones between
    segs, want = [], []
    for k in range(3000):
        n = 0 if k % 7 == 3 else int(rng.integers(1, 3 * E))
        r = rng.normal(0.0, 1.0, n).astype(np.float32).view(np.uint32)
        c = r.copy()
        if n and k % 4 == 0:
            c[rng.integers(0, n, 3)] ^= 0x00400000
        R, C = dev(r, "f32"), dev(c, "f32")
        segs.append((R, C, 1e-6, 0.0, False))
        want.append(_stop_expect(oracle.compare(r, c, "f32", 1e-6, 0.0, False)))
    print("stop-at-first many", len(segs), flush=True)
    for g, w in zip(sv.compare_batched(segs, stop_at_first=True), want):
        same_report(g, w)


def test_stop_at_first_words_from_2_32_checks_ago_count_for_nothing(oracle):
    # The words carry the low 32 bits of their check's sequence number.  A check
    # 2^32 numbers after one that posted a mismatch at tile 0 has the same tag:
    # the words must have been cleared in between, or its waves would stop at
    # tile 0 of a segment that passes.  Also across a boundary taken by a plain
    # check, and back to a smaller number.
    L = sv.lib()
    rng = np.random.default_rng(36)
    n = 1 << 22
    ref = rng.normal(0.0, 1.0, n).astype(np.float32).view(np.uint32)
    bad, near = ref.copy(), ref ^ np.uint32(1)
    bad[5] ^= 0x00400000                                         # a mismatch in tile 0
    R, B, N = dev(ref, "f32"), dev(bad, "f32"), dev(near, "f32")
    want_bad = _stop_expect(oracle.compare(ref, bad, "f32", 1e-6, 0.0, False))
    want_near = oracle.compare(ref, near, "f32", 1e-6, 0.0, False)
    assert want_bad["first_mismatch"] == 5 and want_near["mismatches"] == 0 and want_near["err_sum"] > 0
    fail, clean = [(R, B, 1e-6, 0.0, False)], [(R, N, 1e-6, 0.0, False)]
    print("stop-at-first tags", flush=True)
    for before, after, plain_between in ((9, (1 << 32) + 9, False), ((1 << 32) - 3, (2 << 32) - 3, True),
                                         ((3 << 32) + 100, 100, False), (500, 500, False)):   # same number again
        assert L.sv_testing_set_sequence(before) == 0
        same_report(sv.compare_batched(fail, stop_at_first=True)[0], want_bad)       # posts tile 0
        assert L.sv_testing_set_sequence(after) == 0
        if plain_between:                                        # a plain check takes the next number
            same_report(sv.compare(R, N, 1e-6, 0.0), want_near)
            assert L.sv_testing_set_sequence(after) == 0
        same_report(sv.compare_batched(clean, stop_at_first=True)[0], want_near)    # same tag, cleared
    t = sv.compare_submit(R, N, 1e-6, 0.0)
    assert L.sv_testing_set_sequence(7) == sv.SV_ERR_INVALID_ARG                 # a check is pending
    same_report(t.wait(), want_near)


def test_package_imported_before_torch_shares_torchs_runtime():
    """Regression: the package imported before torch used to load the
    system's HIP runtime beside torch's, and every call then failed with "no
    ROCm-capable device"; the binding now loads torch first."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = ("import paper_2609_00058_amd as sv\nimport torch\n"
            "x = torch.zeros(1000, device='cuda')\ny = x.clone(); y[7] = 1.0\n"
            "r = sv.compare(x, y, 0.0, 0.0)\nprint(r['mismatches'], r['first_mismatch'])\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    assert r.stdout.split() == ["1", "7"], r.stdout

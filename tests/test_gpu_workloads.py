"""The five synthetic workloads at full size, in the launch configuration the
benchmark times, against the CPU oracle.

Where the oracle finishes in seconds (chunked over host threads) it runs in
full and the GPU must match it bit for bit (sum within 1e-12 relative); for
the 2 GiB and 4 GiB workloads it checks sampled elements one by one plus
whole segments, and the reports are pinned by closed forms and by the
oracle's class counts.
"""
import numpy as np
import pytest
import torch

import paper_2609_00058_amd as sv
import workloads as W
from gpu_run import bits, bits_at, gpu_cand, gpu_ref, same_report
from oracle_run import (oracle_case, oracle_case_parallel, oracle_elements, special_counts_parallel)

pytestmark = pytest.mark.gpu


def test_uniform_small_full(oracle):
    case = W.uniform_small().cases[0]
    ref = gpu_ref(case.ref)
    cand = gpu_cand(case, ref)
    r, c, want = oracle_case(case)
    assert np.array_equal(bits(ref), r) and np.array_equal(bits(cand), c)
    got = sv.compare(ref, cand, case.rtol, case.atol, case.equal_nan)
    same_report(got, want)
    assert got["mismatches"] == 7


def test_normal_ulp_full(oracle):
    case = W.normal_ulp().cases[0]
    print("normal 2^26: gpu", flush=True)
    ref = gpu_ref(case.ref)
    cand = gpu_cand(case, ref)
    got = sv.compare(ref, cand, case.rtol, case.atol, case.equal_nan)
    print("normal 2^26: oracle", flush=True)
    r, c, want = oracle_case_parallel(case)
    assert np.array_equal(bits(ref), r)
    assert np.array_equal(bits(cand), c)
    same_report(got, want)
    assert got["nan_cand"] == 16 and got["inf_cand"] == 16 and got["mismatches"] >= 32


def test_bf16_batch_full(oracle):
    wl = W.bf16_batch()
    refs, cands = [], []
    print("bf16 batch: gpu", flush=True)
    for case in wl.cases:
        r = gpu_ref(case.ref)
        refs.append(r)
        cands.append(gpu_cand(case, r))
    segs = [(r, c, case.rtol, case.atol, case.equal_nan) for r, c, case in zip(refs, cands, wl.cases)]
    got = sv.compare_batched(segs)
    for rep in got:   # |a - y| <= 2^-7 |y| < atol + rtol |y|: clean by construction
        assert rep["mismatches"] == 0 and rep["first_mismatch"] == -1 and rep["max_rel_err"] <= 2.0 ** -7
    for k in (0, 37, 63):
        print("bf16 batch: oracle segment", k, flush=True)
        r, c, want = oracle_case_parallel(wl.cases[k])
        assert np.array_equal(bits(refs[k]), r) and np.array_equal(bits(cands[k]), c)
        same_report(got[k], want)
    rng = np.random.default_rng(5)
    for k in rng.choice(64, 8, replace=False):
        idx = rng.integers(0, wl.cases[k].ref.n, 2000)
        r, c = oracle_elements(wl.cases[k], idx)
        assert np.array_equal(bits_at(refs[k], idx), r) and np.array_equal(bits_at(cands[k], idx), c)
    del refs, cands, segs
    torch.cuda.empty_cache()


def test_ragged_batch_full(oracle):
    wl = W.ragged_batch()
    print("ragged batch: gpu", flush=True)
    refs = [gpu_ref(c.ref) for c in wl.cases]
    cands = [gpu_cand(c, r) for c, r in zip(wl.cases, refs)]
    got = sv.compare_batched([(r, c, k.rtol, k.atol, k.equal_nan) for r, c, k in zip(refs, cands, wl.cases)])
    faults = wl.expect["faults"]
    print("ragged batch: oracle", flush=True)
    for k, case in enumerate(wl.cases):
        r, c, want = oracle_case_parallel(case)
        assert np.array_equal(bits(refs[k]), r), k
        assert np.array_equal(bits(cands[k]), c), k
        same_report(got[k], want)
        if k in faults:
            assert got[k]["mismatches"] == 1 and got[k]["first_mismatch"] == faults[k]
        else:
            assert got[k]["mismatches"] == 0
    del refs, cands
    torch.cuda.empty_cache()


def test_special_stream_full(oracle):
    wl = W.special_stream()
    case = wl.cases[0]
    print("special 2^30: gpu", flush=True)
    ref = gpu_ref(case.ref)
    cand = gpu_cand(case, ref)
    got = sv.compare(ref, cand, case.rtol, case.atol, case.equal_nan)
    print("special 2^30: oracle class counts", flush=True)
    counts = special_counts_parallel(case.ref)
    assert got["mismatches"] == 0 and got["first_mismatch"] == -1
    assert got["max_abs_err"] == 0.0 and got["max_rel_err"] == 0.0 and got["err_sum"] == 0.0
    assert got["nan_ref"] == got["nan_cand"] == counts[0]
    assert got["inf_ref"] == got["inf_cand"] == counts[1]
    rng = np.random.default_rng(6)
    idx = np.concatenate([np.arange(2048), case.ref.n - 1 - np.arange(2048), rng.integers(0, case.ref.n, 20000)])
    r, c = oracle_elements(case, idx)
    assert np.array_equal(bits_at(ref, idx), r) and np.array_equal(bits_at(cand, idx), c)
    del ref, cand
    torch.cuda.empty_cache()


def test_candidates_round_full(oracle):
    wl = W.candidates_round()
    uniq, which = wl.ref_groups()
    print("candidates round: gpu", flush=True)
    refs = [gpu_ref(s) for s in uniq]
    cands = [gpu_cand(c, refs[j]) for c, j in zip(wl.cases, which)]
    segs = [(refs[j], c, k.rtol, k.atol, k.equal_nan) for c, k, j in zip(cands, wl.cases, which)]
    stop = sv.compare_batched(segs, stop_at_first=True)
    full = sv.compare_batched(segs)
    for k, case in enumerate(wl.cases):
        g = k % 3
        if g == 0:
            assert full[k]["mismatches"] == 0 and full[k]["err_sum"] == 0.0 and stop[k] == full[k]
            continue
        f = full[k]["first_mismatch"]
        assert stop[k]["mismatches"] == 1 and stop[k]["first_mismatch"] == f and stop[k]["err_sum"] == 0.0
        if g == 2:
            assert full[k]["mismatches"] == 1 and f == wl.expect["faults"][k]
        else:
            assert full[k]["mismatches"] > 0.99 * case.ref.n
        # the first mismatch is exact: the oracle, element by element up to it, finds nothing earlier
        lo = 0 if f < 4096 else f - 64
        idx = np.arange(lo, f + 1, dtype=np.uint64)
        r, c = oracle_elements(case, idx)
        assert np.array_equal(bits_at(refs[which[k]], idx), r) and np.array_equal(bits_at(cands[k], idx), c)
        rep = oracle.compare(r, c, "f32", case.rtol, case.atol, case.equal_nan)
        assert rep["first_mismatch"] == f - lo
    print("candidates round: oracle on two whole segments", flush=True)
    for k in (1, 5):
        r, c, want = oracle_case_parallel(wl.cases[k])
        same_report(full[k], want)
    del refs, cands, segs
    torch.cuda.empty_cache()

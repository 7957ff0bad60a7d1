"""The synthetic workloads at full size against the CPU oracle, synthesized
and checked by the same calls the benchmark times.

Single tensors are synthesized with sv_synth and checked with sv_compare; the
batched workloads are synthesized with one sv_synth_batched over the
benchmark's job list (at these sizes 32 vectors per thread in a tile: the lean
32-bit loop of the batched kernel) and checked with one submitted batched
check.  What is compared, bit for bit (the fp64 error sum within 1e-12
relative):
  - uniform_small, normal_ulp: every element of reference and candidate, the report;
  - bf16_batch: every element of all 64 references and candidates, three reports;
  - ragged_batch: every element of all 256 references and candidates, all reports;
  - special_stream: every element of the 2^30-element reference and candidate,
    streamed through the oracle in windows; the report against the oracle's
    class counts and closed form (zero errors);
  - candidates_round: the first mismatch of every failing segment and two
    whole reports.
The oracle runs chunked over host threads (the serial oracle on windows).
A batched synthesis job whose Philox counters pass 2^32 (outside the lean
loop) is checked on sampled elements and against the single-tensor kernel.
"""
import numpy as np
import pytest
import torch

import paper_2609_00058_amd as sv
import workloads as W
from gpu_run import bits, bits_at, empty, gpu_cand, gpu_ref, same_report
from oracle_run import (oracle_case, oracle_case_parallel, oracle_cand_parallel, oracle_elements,
                        oracle_ref_parallel, special_counts_parallel, windowed)

pytestmark = pytest.mark.gpu


def bench_synth(wl):
    """The references of a batched workload, synthesized as the benchmark does:
    one sv_synth_batched over the distinct reference tensors."""
    uniq, which = wl.ref_groups()
    refs = [empty(s.n, s.dtype) for s in uniq]
    sv.synth_batched(sv.SynthBatch([(r, s.seed, s.stream, s.dist, s.params) for s, r in zip(uniq, refs)]))
    return refs, which


def bench_check(wl, refs, which, cands):
    batch = sv.SegmentBatch([(refs[j], c, k.rtol, k.atol, k.equal_nan) for c, k, j in zip(cands, wl.cases, which)])
    return sv.compare_batched_submit(batch, stop_at_first=wl.stop_at_first).wait()


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
    print("bf16 batch: gpu", flush=True)
    refs, which = bench_synth(wl)
    cands = [gpu_cand(case, refs[j]) for case, j in zip(wl.cases, which)]
    got = bench_check(wl, refs, which, cands)
    for rep in got:   # |a - y| <= 2^-7 |y| < atol + rtol |y|: clean by construction
        assert rep["mismatches"] == 0 and rep["first_mismatch"] == -1 and rep["max_rel_err"] <= 2.0 ** -7
    for k, case in enumerate(wl.cases):
        print("bf16 batch: oracle tensor", k, flush=True)
        r = oracle_ref_parallel(case.ref)
        assert np.array_equal(bits(refs[which[k]]), r), k
        c = oracle_cand_parallel(case, r)
        assert np.array_equal(bits(cands[k]), c), k
        if k in (0, 37, 63):
            same_report(got[k], oracle.compare(r, c, case.ref.dtype, case.rtol, case.atol, case.equal_nan))
    del refs, cands
    torch.cuda.empty_cache()


def test_ragged_batch_full(oracle):
    wl = W.ragged_batch()
    print("ragged batch: gpu", flush=True)
    refs, which = bench_synth(wl)
    cands = [gpu_cand(c, refs[j]) for c, j in zip(wl.cases, which)]
    got = bench_check(wl, refs, which, cands)
    faults = wl.expect["faults"]
    print("ragged batch: oracle", flush=True)
    for k, case in enumerate(wl.cases):
        r, c, want = oracle_case_parallel(case)
        assert np.array_equal(bits(refs[which[k]]), r), k
        assert np.array_equal(bits(cands[k]), c), k
        same_report(got[k], want)
        if k in faults:
            assert got[k]["mismatches"] == 1 and got[k]["first_mismatch"] == faults[k]
        else:
            assert got[k]["mismatches"] == 0
    del refs, cands
    torch.cuda.empty_cache()


def test_batched_job_with_counters_past_2_pow_32(oracle):
    """An int32 job of 2^33 + 2^20 elements (two per Philox block): its block
    indices pass 2^32, so the batched kernel takes its general 64-bit loop;
    batched beside a small job as a second tile size would."""
    n = (1 << 33) + (1 << 20)
    params = dict(lo=-(1 << 20), hi=1 << 20)
    big = empty(n, "i32")
    small = empty(1000, "f32")
    print("counters past 2^32: batched synthesis of 32 GiB", flush=True)
    sv.synth_batched([(big, 3, 9, "int_range", params), (small, 3, 10, "normal", dict(mean=5.0, std=10.0))])
    p = oracle.dist_params(**params)
    rng = np.random.default_rng(33)
    edge = np.arange((1 << 33) - 4096, (1 << 33) + 4096, dtype=np.uint64)
    idx = np.concatenate([edge, np.arange(n - 2048, n, dtype=np.uint64), np.arange(2048, dtype=np.uint64),
                          rng.integers(0, n, 50000).astype(np.uint64)])
    assert np.array_equal(bits_at(big, idx), oracle.synth_at(3, 9, "i32", "int_range", p, idx))
    assert np.array_equal(bits(small), oracle.synth(3, 10, "f32", "normal", oracle.dist_params(mean=5.0, std=10.0),
                                                    1000))
    print("counters past 2^32: single-tensor kernel", flush=True)
    one = empty(n, "i32")
    sv.synth(one, 3, 9, "int_range", **params)
    assert torch.equal(one, big)
    del big, one
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
    # every element of reference and candidate, 2^26 at a time
    for off, m in windowed(case.ref.n, 1 << 26):
        print("special 2^30: oracle window at", off, flush=True)
        r = oracle_ref_parallel(case.ref, off, m)
        assert np.array_equal(bits(ref[off:off + m]), r), off
        c = oracle_cand_parallel(case, r, off)
        assert np.array_equal(bits(cand[off:off + m]), c), off
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

"""End-to-end closed-form pins of the oracle on the five synthetic workloads.

Each workload's report is fixed by arithmetic that does not need an
implementation: where the perturbations land relative to the tolerance of
Eq. (1), how many faults were planted, and which classes of special values
were drawn.  The large workloads run at reduced sizes with the same recipe.
"""
import math

import numpy as np

import workloads as W
from oracle_run import oracle_case, oracle_ref


def f32(bits):
    return np.asarray(bits, dtype=np.uint32).view(np.float32)


def test_workloads_are_deterministic_and_sized():
    a, b = W.ragged_batch(), W.ragged_batch()
    assert [c.ref.n for c in a.cases] == [c.ref.n for c in b.cases]
    sizes = np.array([c.ref.n for c in a.cases])
    assert len(a.cases) == 256 and sizes.min() >= 1000 and sizes.max() <= 10 ** 7
    assert len(a.expect["faults"]) == 13
    assert W.uniform_small().total_elems == 65536
    assert W.normal_ulp().total_elems == 1 << 26
    assert W.bf16_batch().total_elems == 64 * 4096 * 4096
    assert W.special_stream().total_elems == 1 << 30
    assert np.array_equal(W.uniform_small().cases[0].steps[1].idx, W.uniform_small().cases[0].steps[1].idx)


def test_uniform_small_reports_the_seven_faults():
    wl = W.uniform_small()
    case = wl.cases[0]
    _, _, rep = oracle_case(case)
    # |delta| ~ 1e-3 > 1e-8 + 1e-5 |y| <= 1.001e-5 at every planted index, zero elsewhere
    assert rep["mismatches"] == 7
    assert rep["first_mismatch"] == wl.expect["first"]
    assert abs(rep["max_abs_err"] - 1e-3) <= 1.2e-7
    assert rep["nan_ref"] == rep["nan_cand"] == rep["inf_ref"] == rep["inf_cand"] == 0


def test_normal_ulp_reports_exactly_the_special_injections():
    wl = W.normal_ulp(1 << 18)
    case = wl.cases[0]
    ref, cand, rep = oracle_case(case)
    # one ulp <= 2^-23 |y| < 1e-6 |y|: every ulp step passes unless it moved an exact zero
    zero_moved = np.nonzero((f32(ref) == 0) & (ref != cand))[0]
    assert rep["mismatches"] == 32 + zero_moved.size
    idx = np.concatenate([case.steps[1].idx, case.steps[2].idx]).astype(np.int64)
    assert rep["first_mismatch"] == int(np.concatenate([idx, zero_moved]).min())
    assert rep["nan_cand"] == 16 and rep["inf_cand"] == 16
    assert rep["nan_ref"] == 0 and rep["inf_ref"] == 0
    assert rep["max_rel_err"] <= 2.0 ** -23
    changed = np.sum(ref != cand) - 32
    p = 1e-3
    assert abs(changed - ref.size * p) < 5 * math.sqrt(ref.size * p)


def test_bf16_batch_has_no_mismatch_and_bounded_error():
    wl = W.bf16_batch(count=3, rows=128, cols=256)
    for case in wl.cases:
        _, _, rep = oracle_case(case)
        # |a - y| <= 2^-9 |y| + half a bf16 ulp <= 2^-7 |y| < 1e-2 + 1e-2 |y|
        assert rep["mismatches"] == 0 and rep["first_mismatch"] == -1
        assert rep["max_rel_err"] <= 2.0 ** -7
        assert rep["max_abs_err"] <= 4 * 2.0 ** -7


def test_ragged_batch_faults_are_found_exactly():
    wl = W.ragged_batch(count=40, lo_exp=2.0, hi_exp=4.0, fault_frac=0.25)
    faults = wl.expect["faults"]
    assert len(faults) == 10
    for k, case in enumerate(wl.cases):
        ref, cand, rep = oracle_case(case)
        if k in faults:
            assert rep["mismatches"] == 1 and rep["first_mismatch"] == faults[k]
        else:
            assert rep["mismatches"] == 0 and rep["first_mismatch"] == -1 and rep["err_sum"] == 0.0
        if case.ref.dtype == "i32":
            v = ref.view(np.int32)
            assert v.min() >= -(1 << 20) and v.max() <= (1 << 20)


def test_special_stream_is_clean_and_counts_classes():
    wl = W.special_stream(1 << 20)
    case = wl.cases[0]
    ref, cand, rep = oracle_case(case)
    # zero sign flips give d = 0; NaN payload changes keep NaN (equal_nan); nothing else moves
    assert rep["mismatches"] == 0 and rep["first_mismatch"] == -1
    assert rep["max_abs_err"] == 0.0 and rep["max_rel_err"] == 0.0 and rep["err_sum"] == 0.0
    x = f32(ref)
    assert rep["nan_ref"] == rep["nan_cand"] == np.isnan(x).sum()
    assert rep["inf_ref"] == rep["inf_cand"] == np.isinf(x).sum()
    n = x.size
    for cnt, p in ((rep["nan_ref"], 0.01), (rep["inf_ref"], 0.005)):
        assert abs(cnt - n * p) < 5 * math.sqrt(n * p)
    assert np.sum((ref != cand) & ((ref & 0x7FFFFFFF) == 0)) > 0
    assert np.sum((ref != cand) & np.isnan(x)) > 0


def test_reference_synthesis_windows_compose():
    case = W.normal_ulp(4096).cases[0]
    full = oracle_ref(case.ref)
    assert np.array_equal(np.concatenate([oracle_ref(case.ref, 0, 1000), oracle_ref(case.ref, 1000)]), full)


def test_candidates_round_verdicts_at_reduced_size():
    from oracle_run import oracle_case
    n = 1 << 14
    wl = W.candidates_round(outputs=2, n=n)
    assert W.candidates_round(outputs=2, n=n).expect == wl.expect and wl.stop_at_first
    uniq, which = wl.ref_groups()
    assert len(uniq) == 2 and which == [0, 0, 0, 1, 1, 1]
    assert wl.synth_bytes == 2 * 4 * n and wl.compare_bytes == 6 * 2 * 4 * n
    for k, case in enumerate(wl.cases):
        _, _, rep = oracle_case(case)
        g = k % 3
        if g == 0:       # reproduces the reference
            assert rep["mismatches"] == 0 and rep["err_sum"] == 0.0 and rep["first_mismatch"] == -1
        elif g == 1:     # |u| <= 1e-2 against rtol 1e-5: wrong almost everywhere
            assert rep["mismatches"] > 0.99 * n and rep["first_mismatch"] < 100
        else:            # exactly the seeded fault
            assert rep["mismatches"] == 1 and rep["first_mismatch"] == wl.expect["faults"][k]

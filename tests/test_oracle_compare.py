"""Pins of the oracle's elementwise check, Eq. (1) of Sec. 4.2.1, and its report.

Eq. (1): V(K, x, y) = I[ |K(x) - y| <= atol + rtol |y| ], with y the reference
output; rtol scales |y| only, so the rule is asymmetric.  The paper does not
say what happens with NaN or infinities; the reading used is numpy's isclose
convention (identical infinities agree; NaN agrees with NaN only when
equal_nan is set), with the decision evaluated in float64.

Pins: exact rational evaluation of Eq. (1) on a brute-force grid of special
values, numpy.isclose on random data, math.fsum for the error sum, numpy max
for the maxima, and closed forms (rtol = atol = 0 means exact equality).
"""
import math
from fractions import Fraction

import numpy as np
import pytest

GRID = [0x00000000, 0x80000000, 0x00000001, 0x80000001, 0x00800000, 0x80800000,
        0x3F800000, 0xBF800000, 0x3F800001, 0x3F7FFFFF, 0x7F7FFFFF, 0xFF7FFFFF,
        0x7F800000, 0xFF800000, 0x7FC00000, 0x7FC00001, 0xFFC12345, 0x7F800001,
        0x3A83126F, 0x00400000]
TOLS = [(0.0, 0.0), (1e-5, 1e-8), (1e-2, 1e-2), (0.5, 0.0), (0.0, 2.0 ** -149), (1e-7, 0.0),
        (1.0, 1e-45), (2.0 ** -23, 0.0)]


def f32(bits):
    return np.asarray(bits, dtype=np.uint32).view(np.float32)


def exact_decision(a, b, rtol, atol, equal_nan):
    if math.isnan(a) or math.isnan(b):
        return equal_nan and math.isnan(a) and math.isnan(b)
    if math.isinf(a) or math.isinf(b):
        return a == b
    return abs(Fraction(a) - Fraction(b)) <= Fraction(atol) + Fraction(rtol) * abs(Fraction(b))


def near_tie(a, b, rtol, atol):
    if not (math.isfinite(a) and math.isfinite(b)):
        return False
    d = abs(Fraction(a) - Fraction(b))
    t = Fraction(atol) + Fraction(rtol) * abs(Fraction(b))
    return abs(d - t) <= Fraction(2) ** -50 * max(d, t)


def test_brute_force_grid_against_exact_rationals(oracle):
    vals = f32(np.array(GRID, dtype=np.uint32))
    ties = []
    for rtol, atol in TOLS:
        for eqn in (False, True):
            for i, a in enumerate(vals):
                for j, b in enumerate(vals):
                    rep = oracle.compare(np.array([GRID[j]], np.uint32), np.array([GRID[i]], np.uint32),
                                         "f32", rtol, atol, eqn)
                    want = exact_decision(float(a), float(b), rtol, atol, eqn)
                    got = rep["mismatches"] == 0
                    if got != want:
                        assert near_tie(float(a), float(b), rtol, atol), (hex(GRID[i]), hex(GRID[j]), rtol, atol)
                        ties.append((rtol, atol, float(a), float(b), got))
                    assert rep["first_mismatch"] == (-1 if got else 0)
    # The only float64-vs-exact differences on this grid: rtol = 1 with |K(x)| far below
    # ulp(|y|) and y of the other sign, where d = |a - y| and t = atol + |y| both round to |y|
    # in float64; exactly, d exceeds t by |a| - atol > 0.  Float64 accepts, exact rejects.
    assert len(ties) == 42
    for rtol, atol, a, b, got in ties:
        assert rtol == 1.0 and atol == 1e-45 and got and abs(a) < abs(b) * 2.0 ** -52 and a * b < 0


def test_zero_tolerance_is_exact_equality_and_no_flush_to_zero(oracle):
    # denormal vs a different denormal must mismatch at rtol = atol = 0 (catches FTZ)
    ref = np.array([1, 0x00000002, 0, 0x80000000, 0x3F800000], np.uint32)
    cand = np.array([2, 0x00000002, 0x80000000, 0, 0x3F800001], np.uint32)
    rep = oracle.compare(ref, cand, "f32", 0.0, 0.0, False)
    assert rep["mismatches"] == 2 and rep["first_mismatch"] == 0
    assert rep["max_abs_err"] == 2.0 ** -23


def _random_pair(rng, n, special_frac=0.05):
    ref = rng.normal(5.0, 10.0, n).astype(np.float32)
    noise = rng.normal(0, 1, n) * np.abs(ref) * 10.0 ** rng.uniform(-9, -2, n)
    cand = (ref.astype(np.float64) + noise).astype(np.float32)
    same = rng.random(n) < 0.2
    cand[same] = ref[same]
    specials = f32(np.array([0x7FC00000, 0xFFC00001, 0x7F800000, 0xFF800000, 0, 0x80000000, 1, 0x80000005],
                            np.uint32))
    for arr in (ref, cand):
        k = rng.random(n) < special_frac
        arr[k] = rng.choice(specials, k.sum())
    return ref, cand


@pytest.mark.parametrize("rtol,atol,eqn", [(1e-5, 1e-8, False), (1e-3, 1e-6, True), (0.0, 0.0, True),
                                           (1e-6, 0.0, False)])
def test_bitmap_counts_and_stats_against_numpy(oracle, rtol, atol, eqn):
    rng = np.random.default_rng(12)
    n = 200003
    ref, cand = _random_pair(rng, n)
    rep = oracle.compare(ref.view(np.uint32), cand.view(np.uint32), "f32", rtol, atol, eqn)
    a, b = cand.astype(np.float64), ref.astype(np.float64)
    ok = np.isclose(a, b, rtol=rtol, atol=atol, equal_nan=eqn)
    bad = np.nonzero(~ok)[0]
    assert rep["n"] == n
    assert rep["mismatches"] == bad.size
    assert rep["first_mismatch"] == (int(bad[0]) if bad.size else -1)
    fin = np.isfinite(a) & np.isfinite(b)
    d = np.abs(a[fin] - b[fin])
    assert rep["max_abs_err"] == d.max()
    with np.errstate(divide="ignore", invalid="ignore"):
        rel = np.where(d == 0, 0.0, d / np.abs(b[fin]))
    assert rep["max_rel_err"] == rel.max()
    assert rep["err_sum"] == pytest.approx(math.fsum(d), rel=1e-15, abs=0)
    assert rep["nan_ref"] == np.isnan(b).sum() and rep["nan_cand"] == np.isnan(a).sum()
    assert rep["inf_ref"] == np.isinf(b).sum() and rep["inf_cand"] == np.isinf(a).sum()


def test_relative_error_conventions(oracle):
    ref = np.array([0.0, 0.0, 2.0, -4.0], np.float32)
    cand = np.array([0.0, 1e-30, 3.0, -4.0], np.float32)
    rep = oracle.compare(ref.view(np.uint32), cand.view(np.uint32), "f32", 1e-3, 0.0, False)
    assert rep["max_rel_err"] == math.inf                      # y = 0, d > 0
    assert rep["mismatches"] == 2 and rep["first_mismatch"] == 1
    rep = oracle.compare(ref[[0, 2]].view(np.uint32), ref[[0, 2]].view(np.uint32), "f32", 0.0, 0.0, False)
    assert rep["max_rel_err"] == 0.0 and rep["err_sum"] == 0.0  # y = 0, d = 0


def test_err_sum_against_fsum_on_wide_range(oracle):
    rng = np.random.default_rng(3)
    n = 1 << 20
    ref = (rng.standard_normal(n) * 10.0 ** rng.uniform(-30, 30, n)).astype(np.float32)
    cand = (ref.astype(np.float64) * (1 + rng.normal(0, 1e-3, n))).astype(np.float32)
    rep = oracle.compare(ref.view(np.uint32), cand.view(np.uint32), "f32", 1e-5, 0.0, False)
    d = np.abs(cand.astype(np.float64) - ref.astype(np.float64))
    assert rep["err_sum"] == pytest.approx(math.fsum(d), rel=1e-15, abs=0)


def test_bf16_values_upcast_exactly(oracle):
    rng = np.random.default_rng(5)
    ref = rng.integers(0, 1 << 16, 50000, dtype=np.uint32).astype(np.uint16)
    cand = (ref.astype(np.int32) + rng.integers(-2, 3, ref.size)).astype(np.uint16)
    rep = oracle.compare(ref, cand, "bf16", 1e-2, 1e-2, True)
    a = f32(cand.astype(np.uint32) << 16).astype(np.float64)
    b = f32(ref.astype(np.uint32) << 16).astype(np.float64)
    ok = np.isclose(a, b, rtol=1e-2, atol=1e-2, equal_nan=True)
    assert rep["mismatches"] == (~ok).sum()
    assert rep["first_mismatch"] == int(np.nonzero(~ok)[0][0])


def test_int32_is_exact_and_ignores_tolerances(oracle):
    ref = np.array([0, 5, -7, 2 ** 31 - 1, -2 ** 31, 100], np.int32)
    cand = np.array([0, 6, -7, -2 ** 31, -2 ** 31, 100], np.int32)
    for rtol, atol in [(0.0, 0.0), (0.5, 10.0)]:
        rep = oracle.compare(ref.view(np.uint32), cand.view(np.uint32), "i32", rtol, atol, False)
        assert rep["mismatches"] == 2 and rep["first_mismatch"] == 1
        assert rep["max_abs_err"] == 2.0 ** 32 - 1
        assert rep["err_sum"] == 1 + 2.0 ** 32 - 1
        assert rep["max_rel_err"] == (2.0 ** 32 - 1) / (2.0 ** 31 - 1)
        assert rep["nan_ref"] == rep["inf_cand"] == 0


def test_empty_and_batched(oracle):
    e = np.empty(0, np.uint32)
    rep = oracle.compare(e, e, "f32", 1e-5, 1e-8, False)
    assert rep == dict(n=0, mismatches=0, first_mismatch=-1, max_abs_err=0.0, max_rel_err=0.0,
                       err_sum=0.0, nan_ref=0, nan_cand=0, inf_ref=0, inf_cand=0)
    rng = np.random.default_rng(9)
    segs = []
    for k, n in enumerate([0, 1, 17, 1000, 4099]):
        ref, cand = _random_pair(rng, n)
        segs.append((ref.view(np.uint32), cand.view(np.uint32), "f32", 1e-4 * (k + 1), 1e-7, k % 2 == 0))
    batch = oracle.compare_batched(segs)
    for s, r in zip(segs, batch):
        assert r == oracle.compare(*s)


def test_invalid_tolerances_rejected(oracle):
    x = np.zeros(4, np.uint32)
    for rtol, atol in [(-1e-5, 0.0), (0.0, -1.0), (math.nan, 0.0), (math.inf, 0.0)]:
        with pytest.raises(oracle.OracleError):
            oracle.compare(x, x, "f32", rtol, atol, False)


def test_integer_types_ignore_the_tolerances_entirely(oracle):
    """Integer elements agree only when equal: the tolerances play no part, and
    values that a float check refuses (negative, NaN, infinite) are not refused
    either; the report is the one of rtol = atol = 0."""
    y = np.array([5, -7, 2 ** 31 - 1, 0], np.int32).view(np.uint32)
    a = np.array([5, -6, 2 ** 31 - 1, 3], np.int32).view(np.uint32)
    want = oracle.compare(y, a, "i32", 0.0, 0.0, False)
    assert want["mismatches"] == 2 and want["first_mismatch"] == 1
    for rtol, atol in [(-1e-5, 0.0), (0.0, -1.0), (math.nan, 0.0), (0.0, math.inf), (1e300, 1e300)]:
        assert oracle.compare(y, a, "i32", rtol, atol, False) == want


# The largest finite fp64 value plus half an ulp: every exact real at or above
# it rounds to +Inf under round-to-nearest-even.
OVERFLOW_AT = Fraction(2) ** 1024 - Fraction(2) ** 970


def test_err_sum_overflow_is_inf(oracle):
    """An fp64 error sum whose exact value passes the overflow threshold is +Inf
    (every d is >= 0, so no summation order brings it back), never NaN; a
    difference that overflows by itself (both values finite) makes d, the
    maxima and the sum +Inf.  Pinned by exact rationals."""
    cases = [
        ([1e308], [-1e308]),                            # d itself overflows
        ([1e308, 1e308], [-7e307, -7e307]),             # each d finite, the total overflows
        ([1.5e308, 0.0, 1.0], [0.0, 1.5e308, 2.0]),     # overflow at the second term, finite terms after
        ([1e308, 5.0], [0.0, 5.0]),                     # near the edge, finite: a check that stays finite
    ]
    for ref, cand in cases:
        y = np.array(ref, np.float64)
        a = np.array(cand, np.float64)
        rep = oracle.compare(y.view(np.uint64), a.view(np.uint64), "f64", 1e-7, 0.0, False)
        exact = [abs(Fraction(float(p)) - Fraction(float(q))) for p, q in zip(cand, ref)]
        total = sum(exact)
        assert not math.isnan(rep["err_sum"])
        if total >= OVERFLOW_AT:
            assert rep["err_sum"] == math.inf
        else:
            assert rep["err_sum"] == float(total)
        dmax = max(exact)
        assert rep["max_abs_err"] == (math.inf if dmax >= OVERFLOW_AT else float(dmax))
        if dmax >= OVERFLOW_AT:
            assert rep["max_rel_err"] == math.inf

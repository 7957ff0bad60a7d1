"""Property-based pins of the oracle (hypothesis, derandomized so every run
draws the same examples).

Eq. (1) of Sec. 4.2.1 on short arrays seeded with special values, in fp32,
fp64 and int32, against exact rational arithmetic: the decision of each pair
(where d and t are within the rounding of an fp64 evaluation of each -- 2^-50
relative, a few units of the smallest subnormal, or both past the overflow
threshold -- the pair is a tie that evaluation may decide either way), the
count and first index, the maxima (fp64 roundings of exact values), the fsum
of the differences, and the NaN / Inf counts per side; and the synthesis windows, which must be slices
of one tensor whatever the offset, length, type or distribution.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings, strategies as st

SETTINGS = dict(max_examples=400, deadline=None, derandomize=True,
                suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])
OVERFLOW_AT = Fraction(2) ** 1024 - Fraction(2) ** 970   # exact values from here round to +Inf in fp64

F32_SPECIAL = [0x00000000, 0x80000000, 0x00000001, 0x80000001, 0x007FFFFF, 0x00800000, 0x3F800000,
               0xBF800000, 0x7F7FFFFF, 0xFF7FFFFF, 0x7F800000, 0xFF800000, 0x7FC00000, 0xFFC00001,
               0x7F800001]
F64_SPECIAL = [0x0, 0x8000000000000000, 0x1, 0x8000000000000001, 0x000FFFFFFFFFFFFF, 0x0010000000000000,
               0x3FF0000000000000, 0xBFF0000000000000, 0x7FEFFFFFFFFFFFFF, 0xFFEFFFFFFFFFFFFF,
               0x7FF0000000000000, 0xFFF0000000000000, 0x7FF8000000000000, 0xFFF8000000000001]


def _pairs(special, width):
    top = (1 << width) - 1
    raw = st.integers(0, top)
    value = st.one_of(st.sampled_from(special), raw)
    # a candidate close to its reference: the same bits moved by a few units in the last place
    near = st.tuples(value, st.integers(-3, 3)).map(lambda t: (t[0], (t[0] + t[1]) & top))
    any_pair = st.tuples(value, value)
    return st.lists(st.one_of(near, any_pair), min_size=0, max_size=24)


TOL = st.tuples(st.one_of(st.sampled_from([0.0, 1e-7, 1e-5, 1e-2, 0.5, 1.0]), st.floats(0.0, 2.0)),
                st.one_of(st.sampled_from([0.0, 1e-45, 1e-8, 1e-2, 2.0]), st.floats(0.0, 4.0)),
                st.booleans())


def _exact(x):
    return Fraction(x)


def _rounded(q):
    """fp64 rounding (to nearest even) of the non-negative exact rational q."""
    return math.inf if q >= OVERFLOW_AT else float(q)


def _expected(ys, xs, rtol, atol, eqn):
    """Exact-rational expectations for reference values ys and candidate values xs (Python floats)."""
    bad, tie = [], []
    maxabs, maxrel, terms = 0.0, 0.0, []
    for y, a in zip(ys, xs):
        if math.isnan(y) or math.isnan(a):
            bad.append(not (eqn and math.isnan(y) and math.isnan(a)))
            tie.append(False)
            continue
        if math.isinf(y) or math.isinf(a):
            bad.append(a != y)
            tie.append(False)
            continue
        d = abs(_exact(a) - _exact(y))
        t = Fraction(atol) + Fraction(rtol) * abs(_exact(y))
        bad.append(not d <= t)
        # the fp64 evaluation rounds d and t once or twice each: it may decide either way within 2^-50
        # relative, within a few units of the smallest subnormal, or where both round to +Inf
        tie.append(abs(d - t) <= Fraction(2) ** -50 * max(d, t) + Fraction(2) ** -1072
                   or (d >= OVERFLOW_AT and Fraction(rtol) * abs(_exact(y)) >= OVERFLOW_AT / 2))
        dr = _rounded(d)
        terms.append(dr)
        maxabs = max(maxabs, dr)
        rel = 0.0 if dr == 0 else (math.inf if y == 0 or math.isinf(dr) else dr / abs(y))
        maxrel = max(maxrel, rel)
    return bad, tie, maxabs, maxrel, terms


def _check_report(rep, ys, xs, rtol, atol, eqn):
    bad, tie, maxabs, maxrel, terms = _expected(ys, xs, rtol, atol, eqn)
    sure = [b and not t for b, t in zip(bad, tie)]
    maybe = [b or t for b, t in zip(bad, tie)]
    assert sum(sure) <= rep["mismatches"] <= sum(maybe)
    if not any(tie):
        assert rep["mismatches"] == sum(bad)
        assert rep["first_mismatch"] == (bad.index(True) if any(bad) else -1)
    elif rep["first_mismatch"] >= 0:
        assert maybe[rep["first_mismatch"]] and not any(sure[:rep["first_mismatch"]])
    assert rep["max_abs_err"] == maxabs
    assert rep["max_rel_err"] == maxrel
    total = sum(Fraction(t) for t in terms if not math.isinf(t))
    if any(math.isinf(t) for t in terms) or total >= OVERFLOW_AT:
        assert rep["err_sum"] == math.inf
    else:
        assert rep["err_sum"] == pytest.approx(math.fsum(terms), rel=1e-15, abs=0)
    assert rep["nan_ref"] == sum(math.isnan(y) for y in ys)
    assert rep["nan_cand"] == sum(math.isnan(a) for a in xs)
    assert rep["inf_ref"] == sum(math.isinf(y) for y in ys)
    assert rep["inf_cand"] == sum(math.isinf(a) for a in xs)
    assert rep["n"] == len(ys)


@settings(**SETTINGS)
@given(pairs=_pairs(F32_SPECIAL, 32), tol=TOL)
def test_f32_check_against_exact_rationals(oracle, pairs, tol):
    rtol, atol, eqn = tol
    ref = np.array([p[0] for p in pairs], np.uint32)
    cand = np.array([p[1] for p in pairs], np.uint32)
    rep = oracle.compare(ref, cand, "f32", rtol, atol, eqn)
    _check_report(rep, [float(v) for v in ref.view(np.float32)], [float(v) for v in cand.view(np.float32)],
                  rtol, atol, eqn)


@settings(**SETTINGS)
@given(pairs=_pairs(F64_SPECIAL, 64), tol=TOL)
def test_f64_check_against_exact_rationals(oracle, pairs, tol):
    rtol, atol, eqn = tol
    ref = np.array([p[0] for p in pairs], np.uint64)
    cand = np.array([p[1] for p in pairs], np.uint64)
    rep = oracle.compare(ref, cand, "f64", rtol, atol, eqn)
    _check_report(rep, [float(v) for v in ref.view(np.float64)], [float(v) for v in cand.view(np.float64)],
                  rtol, atol, eqn)


@settings(**SETTINGS)
@given(pairs=st.lists(st.tuples(st.integers(-2 ** 31, 2 ** 31 - 1), st.integers(-2 ** 31, 2 ** 31 - 1)),
                      max_size=24), tol=TOL)
def test_int32_check_is_exact_equality(oracle, pairs, tol):
    rtol, atol, eqn = tol
    ys = [p[0] for p in pairs]
    xs = [p[0] if k % 3 else p[1] for k, p in enumerate(pairs)]     # a third of the pairs differ
    rep = oracle.compare(np.array(ys, np.int32).view(np.uint32), np.array(xs, np.int32).view(np.uint32),
                         "i32", rtol, atol, eqn)
    bad = [a != y for y, a in zip(ys, xs)]
    assert rep["mismatches"] == sum(bad)
    assert rep["first_mismatch"] == (bad.index(True) if any(bad) else -1)
    d = [abs(a - y) for y, a in zip(ys, xs)]
    assert rep["max_abs_err"] == float(max(d, default=0))
    assert rep["err_sum"] == float(sum(d))                        # below 2^53: exact
    rel = [0.0 if e == 0 else (math.inf if y == 0 else float(Fraction(e, abs(y)))) for y, e in zip(ys, d)]
    assert rep["max_rel_err"] == max(rel, default=0.0)


DISTS = [("uniform", "f32", dict(a=-3.0, b=7.0)), ("uniform", "bf16", dict(a=-4.0, b=4.0)),
         ("normal", "f32", dict(mean=5.0, std=10.0)), ("normal", "f16", dict(mean=0.0, std=1.0)),
         ("int_range", "i32", dict(lo=-5, hi=1 << 20)), ("int_range", "u8", dict(lo=3, hi=200)),
         ("int_range", "i64", dict(lo=-(1 << 40), hi=1 << 40)), ("uniform", "f64", dict(a=0.0, b=1.0)),
         ("special", "f32", dict(mean=0.0, std=1e3, p_nan=0.1, p_inf=0.1, p_denorm=0.1, p_zero=0.1)),
         ("special", "bf16", dict(mean=0.0, std=1.0, p_nan=0.2, p_inf=0.0, p_denorm=0.2, p_zero=0.0))]


@settings(**SETTINGS)
@given(case=st.sampled_from(DISTS), seed=st.integers(0, 2 ** 64 - 1), stream=st.integers(0, 2 ** 64 - 1),
       offset=st.one_of(st.integers(0, 100), st.integers(0, 2 ** 44)), n=st.integers(0, 40),
       back=st.integers(0, 9))
def test_synthesis_windows_are_slices(oracle, case, seed, stream, offset, n, back):
    dist, dtype, params = case
    p = oracle.dist_params(**params)
    start = max(offset - back, 0)
    whole = oracle.synth(seed, stream, dtype, dist, p, n + (offset - start), offset=start)
    window = oracle.synth(seed, stream, dtype, dist, p, n, offset=offset)
    assert np.array_equal(window.view(np.uint8), whole[offset - start:].view(np.uint8))
    idx = (np.arange(n, dtype=np.uint64)[::-1] + np.uint64(offset)).astype(np.uint64)
    picked = oracle.synth_at(seed, stream, dtype, dist, p, idx)
    assert np.array_equal(picked.view(np.uint8), np.ascontiguousarray(window[::-1]).view(np.uint8))

"""Pins of the oracle's fp16, fp64, uint8 and int64 paths against numpy and
exact arithmetic (no GPU)."""
import math
from fractions import Fraction

import numpy as np
import pytest


# ------------------------------------------------------------ fp32 -> fp16
def _numpy_f16(bits):
    return np.asarray(bits, np.uint32).view(np.float32).astype(np.float16).view(np.uint16)


def test_f16_rounding_matches_numpy_on_random_and_edge_patterns(oracle):
    rng = np.random.default_rng(16)
    pats = [rng.integers(0, 2 ** 32, 2_000_000, dtype=np.uint64).astype(np.uint32)]
    # every finite half, its midpoints to the next half, and one fp32 ulp either side of them
    h = np.arange(0, 0x7C00, dtype=np.uint16)
    lo = h.view(np.float16).astype(np.float32)
    hi = (h + 1).view(np.float16).astype(np.float32)
    mid = ((lo.astype(np.float64) + hi.astype(np.float64)) / 2).astype(np.float32)   # exact: 12 bits
    for v in (lo, mid):
        b = v.view(np.uint32)
        pats += [b, b + 1, b - 1, b | 0x80000000]
    edges = np.array([65504.0, 65519.996, 65520.0, 65536.0, 1e30, 2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -26,
                      2.0 ** -25 * 1.0000001, 2.0 ** -14, 2.0 ** -14 * (1 - 2 ** -11), 0.0, np.inf],
                     np.float32).view(np.uint32)
    pats += [edges, edges | 0x80000000]
    allp = np.concatenate(pats).astype(np.uint32)
    finite = (allp & 0x7F800000) != 0x7F800000
    assert np.array_equal(oracle.f16_rne_n(allp[finite]), _numpy_f16(allp[finite]))


def test_f16_nan_and_infinity_rules(oracle):
    rng = np.random.default_rng(17)
    nans = (rng.integers(1, 2 ** 23, 100_000).astype(np.uint32) | 0x7F800000)
    nans = np.concatenate([nans, nans | 0x80000000, np.array([0x7F800000, 0xFF800000], np.uint32)])
    got = oracle.f16_rne_n(nans)
    assert np.array_equal(got, _numpy_f16(nans))        # NaN keeps sign and top fraction bits, Inf stays Inf
    assert np.all(np.isnan(got[:-2].view(np.float16)))


# ------------------------------------------------------------ synthesis
def test_f64_uniform_closed_form_and_bounds(oracle):
    n = 20000
    for a, b in [(-1.0, 1.0), (0.0, 4.0), (-3.0, 5.0)]:        # power-of-two spans: a + span U is exact
        p = oracle.dist_params(a=a, b=b)
        got = oracle.synth(3, 4, "f64", "uniform", p, n).view(np.float64)
        w = oracle.philox_blocks(3, 4, 0, n // 2).reshape(-1, 4).astype(np.uint64)
        R = np.stack([(w[:, 1] << 32) | w[:, 0], (w[:, 3] << 32) | w[:, 2]], axis=1).reshape(-1)
        for k in range(0, n, 97):
            want = Fraction(a) + Fraction(b - a) * Fraction(int(R[k]) >> 11, 2 ** 53)
            assert Fraction(float(got[k])) == want
        assert got.min() >= a and got.max() < b
    p = oracle.dist_params(a=-0.3, b=0.7)
    got = oracle.synth(3, 5, "f64", "uniform", p, 200_000).view(np.float64)
    assert got.min() >= -0.3 and got.max() <= 0.7
    assert abs(got.mean() - 0.2) < 5 * math.sqrt(1 / 12 / 200_000)
    # 53 significant random bits: far more distinct values than an fp32 source could give
    assert np.unique(got).size > 199_000


def test_f64_normal_and_special_widen_the_fp32_values(oracle):
    for dist, prm in [("normal", dict(mean=5.0, std=10.0)),
                      ("special", dict(mean=0.0, std=1e3, p_nan=0.2, p_inf=0.1, p_denorm=0.1, p_zero=0.1))]:
        p = oracle.dist_params(**prm)
        f32 = oracle.synth(8, 1, "f32", dist, p, 50_000)
        f64 = oracle.synth(8, 1, "f64", dist, p, 50_000)
        fin = (f32 & 0x7F800000) != 0x7F800000
        assert np.array_equal(f64[fin].view(np.float64), f32[fin].view(np.float32).astype(np.float64))
        nf = ~fin                                     # Inf and NaN: sign and fraction carried over bit by bit
        want = ((f32[nf].astype(np.uint64) >> 31) << 63) | 0x7FF0000000000000 | \
               ((f32[nf].astype(np.uint64) & 0x7FFFFF) << 29)
        assert np.array_equal(f64[nf], want)
        f16 = oracle.synth(8, 1, "f16", dist, p, 50_000)
        assert np.array_equal(f16, oracle.f16_rne_n(f32))


def test_integer_ranges_closed_forms(oracle):
    n = 20000
    w = oracle.philox_blocks(6, 2, 0, n // 2).reshape(-1, 4).astype(np.uint64)
    R = np.stack([(w[:, 1] << 32) | w[:, 0], (w[:, 3] << 32) | w[:, 2]], axis=1).reshape(-1)
    # uint8: one 32-bit word per element, word i mod 4 of block i / 4
    w32 = oracle.philox_blocks(6, 2, 0, n // 4).reshape(-1).astype(np.uint64)
    u8 = oracle.synth(6, 2, "u8", "int_range", oracle.dist_params(lo=0, hi=255), n)
    assert np.array_equal(u8, (w32 >> 24).astype(np.uint8))                # range 2^8: the top 8 bits
    u8_16 = oracle.synth(6, 2, "u8", "int_range", oracle.dist_params(lo=100, hi=115), n)
    assert np.array_equal(u8_16, (100 + (w32 >> 28)).astype(np.uint8))     # range 2^4: the top 4 bits
    u8_odd = oracle.synth(6, 2, "u8", "int_range", oracle.dist_params(lo=3, hi=203), n)
    assert u8_odd.tolist() == [3 + ((int(x) * 201) >> 32) for x in w32]   # floor(w * 201 / 2^32)
    full = oracle.synth(6, 2, "i64", "int_range", oracle.dist_params(lo=-2 ** 63, hi=2 ** 63 - 1), n)
    assert np.array_equal(full, R ^ np.uint64(1 << 63))                    # range 2^64: lo + R
    p40 = oracle.synth(6, 2, "i64", "int_range", oracle.dist_params(lo=-(2 ** 39), hi=2 ** 39 - 1), n)
    assert np.array_equal(p40.view(np.int64), (R >> 24).astype(np.int64) - 2 ** 39)
    odd = oracle.synth(6, 2, "i64", "int_range", oracle.dist_params(lo=-7, hi=10 ** 15), n).view(np.int64)
    want = [-7 + ((int(r) * (10 ** 15 + 8)) >> 64) for r in R[:2000]]
    assert odd[:2000].tolist() == want and odd.min() >= -7 and odd.max() <= 10 ** 15
    small = oracle.synth(6, 3, "u8", "int_range", oracle.dist_params(lo=3, hi=9), 70_000)
    counts = np.bincount(small, minlength=10)[3:10]
    assert counts.sum() == 70_000 and np.all(np.abs(counts - 10_000) < 5 * math.sqrt(10_000))
    with pytest.raises(RuntimeError):
        oracle.synth(0, 0, "u8", "int_range", oracle.dist_params(lo=0, hi=256), 4)
    with pytest.raises(RuntimeError):
        oracle.synth(0, 0, "f64", "int_range", oracle.dist_params(lo=0, hi=5), 4)


# ------------------------------------------------------------ Eq. (1) on the new types
def _numpy_report(y, a, rtol, atol, equal_nan):
    fin = np.isfinite(y) & np.isfinite(a)
    close = np.isclose(a, y, rtol=rtol, atol=atol, equal_nan=equal_nan)
    bad = ~close
    d = np.where(fin, np.abs(a - y), 0.0)
    return int(bad.sum()), (int(np.argmax(bad)) if bad.any() else -1), float(d.max(initial=0.0))


@pytest.mark.parametrize("dtype,np_t", [("f16", np.float16), ("f64", np.float64)])
def test_compare_float_types_match_numpy_isclose(oracle, dtype, np_t):
    rng = np.random.default_rng(30)
    n = 50_000
    y = rng.normal(5.0, 10.0, n)
    a = y * (1 + rng.normal(0, 1, n) * 10.0 ** rng.uniform(-8, -1, n))
    sp = np.array([np.nan, np.inf, -np.inf, 0.0, -0.0])
    for arr in (y, a):
        k = rng.random(n) < 0.03
        arr[k] = rng.choice(sp, k.sum())
    y, a = y.astype(np_t), a.astype(np_t)
    yw, aw = y.astype(np.float64), a.astype(np.float64)
    store = np.uint16 if dtype == "f16" else np.uint64
    for rtol, atol, eqn in [(1e-3, 1e-5, False), (1e-2, 0.0, True), (0.0, 0.0, False)]:
        rep = oracle.compare(y.view(store), a.view(store), dtype, rtol, atol, eqn)
        mism, first, maxabs = _numpy_report(yw, aw, rtol, atol, eqn)
        assert (rep["mismatches"], rep["first_mismatch"], rep["max_abs_err"]) == (mism, first, maxabs)
        assert rep["nan_ref"] == int(np.isnan(yw).sum()) and rep["inf_cand"] == int(np.isinf(aw).sum())


def test_compare_int64_is_exact_beyond_2_pow_53(oracle):
    y = np.array([2 ** 60, -2 ** 62, 2 ** 63 - 1, -2 ** 63, 5, 0], np.int64)
    a = y.copy()
    a[0] += 1                                   # equal as fp64, different as integers
    a[2] = -2 ** 63                              # the largest possible difference
    rep = oracle.compare(y.view(np.uint64), a.view(np.uint64), "i64", 0.5, 1e9, False)
    assert rep["mismatches"] == 2 and rep["first_mismatch"] == 0
    assert rep["max_abs_err"] == float(2 ** 64 - 1) == 2.0 ** 64   # |a - y| = 2^64 - 1, rounded once
    assert rep["err_sum"] == 1.0 + 2.0 ** 64
    u = np.array([0, 255, 7], np.uint8)
    rep = oracle.compare(u, np.array([0, 254, 7], np.uint8), "u8", 1.0, 1.0, False)
    assert rep["mismatches"] == 1 and rep["first_mismatch"] == 1 and rep["max_abs_err"] == 1.0


# ------------------------------------------------------------ candidate steps
def test_candidate_steps_on_the_new_types(oracle):
    rng = np.random.default_rng(40)
    f16 = rng.normal(0, 100, 10_000).astype(np.float16)
    f16[:4] = [0.0, -0.0, np.inf, 65504.0]
    c = oracle.perturb(1, 2, "f16", "ulp", f16.view(np.uint16), np.empty(f16.size, np.uint16), p=1.0)
    toward = np.where(c.view(np.float16).astype(np.float64) > f16.astype(np.float64), np.inf, -np.inf)
    assert np.array_equal(c.view(np.float16), np.nextafter(f16, toward.astype(np.float16)))
    f64 = rng.normal(0, 1e10, 10_000)
    c = oracle.perturb(1, 3, "f64", "ulp", f64.view(np.uint64), np.empty(f64.size, np.uint64), p=1.0)
    moved = c.view(np.float64)
    assert np.all(moved != f64)
    assert np.array_equal(moved, np.nextafter(f64, np.where(moved > f64, np.inf, -np.inf)))
    idx = np.array([0, 5, 9999], np.uint64)
    c = oracle.perturb(0, 0, "f64", "fault_at", f64.view(np.uint64), f64.view(np.uint64).copy(), idx=idx)
    assert np.array_equal(c.view(np.float64)[idx], f64[idx] + (1.0 + np.abs(f64[idx])))
    u8 = np.array([255, 3, 0], np.uint8)
    c = oracle.perturb(0, 0, "u8", "fault_at", u8, u8.copy(), idx=np.array([0, 2], np.uint64))
    assert c.tolist() == [0, 3, 1]                       # wraps in 8 bits
    i64 = np.array([2 ** 63 - 1, -1], np.int64).view(np.uint64)
    c = oracle.perturb(0, 0, "i64", "fault_at", i64, i64.copy(), idx=np.array([0, 1], np.uint64))
    assert c.view(np.int64).tolist() == [-2 ** 63, 0]
    c = oracle.perturb(0, 0, "f16", "set_at", f16.view(np.uint16), f16.view(np.uint16).copy(), bits=0x7E00,
                       idx=np.array([7], np.uint64))
    assert c[7] == 0x7E00
    with pytest.raises(RuntimeError):
        oracle.perturb(0, 0, "f64", "scale", f64.view(np.uint64), np.empty(f64.size, np.uint64), p=1.0, value=0.1)

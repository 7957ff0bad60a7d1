"""Pins of the oracle's distribution transforms.

Sec. 4.2.1 asks that test inputs come from a broad numeric range (a Gaussian
with mean 5 and standard deviation 10 is its example).  The transforms below
are conventions the paper leaves open; each is pinned against mathematics
that does not depend on the oracle: exact closed forms, exhaustive error
bounds against float64 / mpmath, special cases, moments and Kolmogorov-Smirnov
statistics, and library routines (torch's bf16 rounding).
"""
import math
import os
import re
from fractions import Fraction

import numpy as np
import pytest
import scipy.stats as st

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def f32(bits):
    return np.asarray(bits, dtype=np.uint32).view(np.float32)


def ulp32(x):
    x = np.abs(np.asarray(x, np.float64))
    e = np.floor(np.log2(np.maximum(x, 2.0 ** -126)))
    return 2.0 ** (e - 23)


def rne32_exact(x):
    """fp32 round-to-nearest-even of an exact value (a Fraction or a float)."""
    fx = Fraction(x)
    lo = np.float32(float(fx))
    cands = [np.nextafter(lo, np.float32(-np.inf)), lo, np.nextafter(lo, np.float32(np.inf))]
    return float(min(cands, key=lambda c: (abs(Fraction(float(c)) - fx), int(np.float32(c).view(np.uint32)) & 1)))


# --------------------------------------------------------------- constants
def _oracle_constants():
    src = open(os.path.join(ROOT, "oracle", "sv_oracle.c")).read()
    return {m.group(1): float.fromhex(m.group(2))
            for m in re.finditer(r"static const float (\w+) = (-?0x[0-9a-fA-F.]+p[-+]?\d+)f;", src)}


def test_transform_constants_are_the_fp32_roundings_of_their_definitions():
    mp = pytest.importorskip("mpmath")
    mp.mp.prec = 300

    def rne32(x):
        # fp32 round-to-nearest-even of an mpf, exactly
        v = float(x)                       # correctly rounded to fp64 first is not enough;
        lo = np.float32(v)                 # so check the neighbours explicitly
        cands = [np.nextafter(lo, np.float32(-np.inf)), lo, np.nextafter(lo, np.float32(np.inf))]
        best = min(cands, key=lambda c: (abs(mp.mpf(float(c)) - x),
                                         int(np.float32(c).view(np.uint32)) & 1))
        return float(best)

    half_pi = mp.pi / 2
    ln2 = mp.log(2)
    ln2_hi = mp.floor(ln2 * 2 ** 16) / 2 ** 16
    want = {"LN_SQRT2": mp.sqrt(2), "LN2_HI": ln2_hi, "LN2_LO": ln2 - ln2_hi}
    # ln(1 + f) / f on [sqrt(1/2) - 1, sqrt(2) - 1]: Chebyshev interpolation at 10 nodes
    lo, hi = mp.sqrt(mp.mpf(1) / 2) - 1, mp.sqrt(2) - 1
    poly = mp.chebyfit(lambda x: mp.log1p(x) / x if x != 0 else mp.mpf(1), [lo, hi], 10)
    assert rne32(poly[-1]) == 1.0
    for k in range(1, 10):
        want["LN_P%d" % k] = poly[9 - k]
    want["SC_B"] = 4 * half_pi / 2 ** 24          # 2 pi / 2^24
    want["SC_S3"] = mp.mpf(-1) / 6                 # sin b = b - b^3 / 6
    got = _oracle_constants()
    assert set(want) <= set(got)
    for name, x in want.items():
        assert got[name] == rne32(x), name
    assert float(ln2_hi) == 45426 / 2 ** 16


# --------------------------------------------------------------- uniform
@pytest.mark.parametrize("a,b", [(-1.0, 1.0), (-4.0, 4.0), (0.0, 1.0)])
def test_uniform_closed_form_on_power_of_two_spans(oracle, a, b):
    # element i = a + (b - a) * k * 2^-24 exactly, k = top 24 bits of word i%4 of block i/4
    n = 4096
    v = f32(oracle.synth(2, 5, "f32", "uniform", oracle.dist_params(a=a, b=b), n))
    w = oracle.philox_blocks(2, 5, 0, n // 4).reshape(-1)
    k = w >> 8
    for i in range(n):
        assert Fraction(float(v[i])) == Fraction(a) + Fraction(b - a) * Fraction(int(k[i]), 2 ** 24)


def test_uniform_half_open_and_moments(oracle):
    n = 1 << 20
    a, b = -3.0, 7.5
    v = f32(oracle.synth(0, 1, "f32", "uniform", oracle.dist_params(a=a, b=b), n)).astype(np.float64)
    assert v.min() >= a and v.max() < b
    mean_sigma = (b - a) / math.sqrt(12 * n)
    assert abs(v.mean() - (a + b) / 2) < 5 * mean_sigma
    var = (b - a) ** 2 / 12
    assert abs(v.var() - var) < 5 * var * math.sqrt(0.8 / n)   # var of sample var: (4/5) var^2 / n
    d = st.kstest(v, "uniform", args=(a, b - a)).statistic
    assert d < 1.95 / math.sqrt(n)


def _bf16_of_exact_fp32(vals):
    """torch's fp32 -> bf16 rounding (round to nearest even) of fp32 values."""
    import torch
    return torch.from_numpy(np.asarray(vals, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _half_words(oracle, seed, stream, n):
    """The 16-bit halves of the Philox words in element order: block c gives
    elements 8c .. 8c + 7 from words 0..3, low half first."""
    w = oracle.philox_blocks(seed, stream, 0, -(-n // 8)).reshape(-1)
    return np.stack([w & 0xFFFF, w >> 16], axis=1).reshape(-1)[:n]


@pytest.mark.parametrize("a,b", [(-4.0, 4.0), (-1.0, 1.0), (0.0, 1.0), (-0.5, 0.25)])
def test_uniform_bf16_closed_form_from_half_words(oracle, a, b):
    """bf16 uniform: element i = RNE_bf16(a + (b - a) k 2^-16) with k the 16-bit
    half-word of element i; on power-of-two spans a + (b - a) k 2^-16 is an fp32
    value exactly (checked with Fractions), so the oracle's two fp32 roundings
    vanish and the result is torch's bf16 rounding of the exact value."""
    n = 1 << 15
    got = oracle.synth(4, 11, "bf16", "uniform", oracle.dist_params(a=a, b=b), n)
    k = _half_words(oracle, 4, 11, n)
    table = np.array([float(Fraction(a) + Fraction(b - a) * Fraction(j, 1 << 16)) for j in range(1 << 16)])
    for j in (0, 1, 12345, (1 << 16) - 1):
        assert Fraction(float(np.float32(table[j]))) == Fraction(a) + Fraction(b - a) * Fraction(j, 1 << 16)
    assert np.array_equal(table.astype(np.float32).astype(np.float64), table)   # every value exact in fp32
    want = _bf16_of_exact_fp32(table.astype(np.float32))[k]
    assert np.array_equal(got, want)


def test_uniform_bf16_general_span_is_rne_of_the_fp32_value(oracle):
    """On a span that is not a power of two: the fp32 value is the rounding of
    a + rounding(span U) (two roundings, checked with Fractions), then bf16."""
    a, b = -3.0, 7.5
    n = 1 << 14
    got = oracle.synth(6, 2, "bf16", "uniform", oracle.dist_params(a=a, b=b), n)
    k = _half_words(oracle, 6, 2, n)
    span = np.float32(b) - np.float32(a)
    v = np.array([rne32_exact(Fraction(a) + Fraction(rne32_exact(Fraction(float(span)) * Fraction(int(j), 1 << 16))))
                  for j in k], np.float32)
    assert np.array_equal(got, _bf16_of_exact_fp32(v))


def test_uniform_bf16_distribution(oracle):
    """2^22 draws on [-4, 4): each bf16 value occurs with the probability the
    65,536 equally likely half-words give it (chi-square), the moments of a
    uniform variable, no correlation between the two halves of a word or
    between neighbouring words, and the bounds (rounding may reach b)."""
    import torch
    a, b = -4.0, 4.0
    n = 1 << 22
    out = oracle.synth(1, 7, "bf16", "uniform", oracle.dist_params(a=a, b=b), n)
    vals = (out.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    assert vals.min() >= a and vals.max() <= b
    exact = np.array([a + (b - a) * j / 65536 for j in range(1 << 16)], np.float32)
    keys = _bf16_of_exact_fp32(exact)
    uk, cnt = np.unique(keys, return_counts=True)
    p = cnt / 65536.0
    assert np.isin(out, uk).all()                           # nothing outside the reachable set
    obs = np.bincount(np.searchsorted(uk, out), minlength=uk.size)
    chi2 = ((obs - n * p) ** 2 / (n * p)).sum()
    dof = uk.size - 1
    assert chi2 < dof + 5 * math.sqrt(2 * dof)
    mean_sigma = (b - a) / math.sqrt(12 * n)
    assert abs(vals.mean() - (a + b) / 2) < 5 * mean_sigma
    for lag in (1, 2):                                      # halves of one word; neighbouring words
        r = np.corrcoef(vals[:-lag], vals[lag:])[0, 1]
        assert abs(r) < 5 / math.sqrt(n)


def test_uniform_bf16_windows_are_slices(oracle):
    p = oracle.dist_params(a=-4.0, b=4.0)
    full = oracle.synth(3, 3, "bf16", "uniform", p, 4096)
    for off in (1, 7, 8, 9, 1001):
        assert np.array_equal(oracle.synth(3, 3, "bf16", "uniform", p, 500, offset=off), full[off:off + 500])
    assert np.array_equal(oracle.synth(3, 3, "bf16", "uniform", p, 100), full[:100])


# --------------------------------------------------------------- ln / sincos / Box-Muller
def test_ln_exhaustive_on_all_box_muller_inputs(oracle):
    # every u1 = k 2^-24, k = 1 .. 2^24, within 1.6 ulp of float64 log (measured max 1.53)
    k = np.arange(1, (1 << 24) + 1, dtype=np.float64)
    u1 = (k * 2.0 ** -24).astype(np.float32)
    got = oracle.ln_f32_n(u1).astype(np.float64)
    want = np.log(u1.astype(np.float64))
    assert got[-1] == 0.0                      # ln 1 = 0 exactly
    nz = want != 0
    err = np.abs(got[nz] - want[nz]) / ulp32(want[nz])
    assert err.max() <= 1.6
    assert np.all(got[:-1] < 0)


def test_ln_at_powers_of_two_is_e_ln2_within_one_ulp(oracle):
    for e in range(-24, 0):
        want = e * math.log(2)
        assert abs(float(oracle.ln_f32(2.0 ** e)) - want) <= float(ulp32(want))


def test_sincos_table_is_the_correctly_rounded_values(oracle):
    """The 256 table values are sin and cos of 2 pi k / 256 rounded to nearest
    fp32 (mpmath at 200 bits), exact zeros positive; symmetric as the
    functions are."""
    mp = pytest.importorskip("mpmath")
    mp.mp.prec = 200
    s, c = oracle.sincos_table()
    for k in range(256):
        x = 2 * mp.pi * k / 256
        for got, v in ((s[k], mp.sin(x)), (c[k], mp.cos(x))):
            if k % 64 == 0 and abs(v) < mp.mpf(2) ** -100:
                assert got == 0.0 and not math.copysign(1.0, float(got)) < 0, k
            else:
                assert float(got) == rne32_exact(Fraction(mp.nstr(v, 80))), k
    assert np.array_equal(s[1:64], c[63:0:-1]) and np.array_equal(s[:128], -s[128:] + 0.0)


def test_sincos_exhaustive(oracle):
    # all 2^24 angles 2 pi j / 2^24 within 2.5 ulp (measured max 2.491), exact at the axes
    j = np.arange(1 << 24, dtype=np.uint32)
    s, c = oracle.sincos_2pi_f32_n(j)
    q = j >> 22
    f = (j & 0x3FFFFF).astype(np.float64) * 2.0 ** -22
    S, C = np.sin(np.pi / 2 * f), np.cos(np.pi / 2 * f)   # quarter-turn reduction is exact
    sref = np.select([q == 0, q == 1, q == 2, q == 3], [S, C, -S, -C])
    cref = np.select([q == 0, q == 1, q == 2, q == 3], [C, -S, -C, S])
    for got, want in ((s, sref), (c, cref)):
        nz = want != 0
        assert np.all(got[~nz] == 0)
        err = np.abs(got[nz].astype(np.float64) - want[nz]) / ulp32(want[nz])
        assert err.max() <= 2.5
        assert (err > 1).mean() < 0.04      # measured 2.9 % above one ulp
    axes = np.array([0, 1 << 22, 2 << 22, 3 << 22], dtype=np.uint32)
    s, c = oracle.sincos_2pi_f32_n(axes)
    assert list(s) == [0.0, 1.0, 0.0, -1.0] and list(c) == [1.0, 0.0, -1.0, 0.0]
    assert np.all(s * s + c * c <= 1.0 + 4e-7)


def test_box_muller_accuracy_and_special_cases(oracle):
    w = oracle.philox_blocks(0, 0, 0, 1 << 17)
    zc = np.empty(w.shape[0]); zs = np.empty(w.shape[0])
    for k in range(w.shape[0]):
        zc[k], zs[k] = oracle.box_muller_f32(int(w[k, 0]), int(w[k, 1]))
    u1 = ((w[:, 0] >> 8).astype(np.float64) + 1) * 2.0 ** -24
    u2 = (w[:, 1] >> 8).astype(np.float64) * 2.0 ** -24
    r = np.sqrt(-2 * np.log(u1))
    for got, want in ((zc, r * np.cos(2 * np.pi * u2)), (zs, r * np.sin(2 * np.pi * u2))):
        nz = np.abs(want) > 1e-30
        assert (np.abs(got[nz] - want[nz]) / ulp32(want[nz])).max() <= 4.5
    # u1 = 1 gives r = 0; u2 = 0 gives (r, 0); the largest radius is sqrt(48 ln 2)
    assert all(z == 0 for z in oracle.box_muller_f32(0xFFFFFFFF, 12345 << 8))
    zc0, zs0 = oracle.box_muller_f32(0, 0)
    assert zs0 == 0.0 and abs(float(zc0) - math.sqrt(48 * math.log(2))) <= 4 * float(ulp32(5.77))


def test_normal_element_order(oracle):
    p = oracle.dist_params(mean=0.0, std=1.0)
    v = f32(oracle.synth(4, 2, "f32", "normal", p, 64))
    w = oracle.philox_blocks(4, 2, 0, 16)
    for c in range(16):
        a = oracle.box_muller_f32(int(w[c, 0]), int(w[c, 1]))
        b = oracle.box_muller_f32(int(w[c, 2]), int(w[c, 3]))
        assert list(v[4 * c:4 * c + 4]) == [a[0], a[1], b[0], b[1]]
    # mean + std z is one fused multiply-add
    p = oracle.dist_params(mean=5.0, std=10.0)
    v = f32(oracle.synth(4, 2, "f32", "normal", p, 64)).astype(np.float64)
    z = f32(oracle.synth(4, 2, "f32", "normal", oracle.dist_params(mean=0.0, std=1.0), 64)).astype(np.float64)
    assert np.array_equal(v, np.array([rne32_exact(Fraction(10) * Fraction(x) + 5) for x in z]))


@pytest.mark.parametrize("mean,std", [(0.0, 1.0), (5.0, 10.0)])
def test_normal_moments_and_ks(oracle, mean, std):
    n = 1 << 20
    v = f32(oracle.synth(0, 7, "f32", "normal", oracle.dist_params(mean=mean, std=std), n)).astype(np.float64)
    z = (v - mean) / std
    assert abs(z.mean()) < 5 / math.sqrt(n)
    assert abs(z.var() - 1) < 5 * math.sqrt(2 / n)
    assert abs(st.skew(z)) < 5 * math.sqrt(6 / n)
    assert abs(st.kurtosis(z)) < 5 * math.sqrt(24 / n)
    assert st.kstest(z, "norm").statistic < 1.95 / math.sqrt(n)
    assert np.abs(z).max() <= math.sqrt(48 * math.log(2)) * (1 + 1e-6)


# --------------------------------------------------------------- integer range
def test_int_range_power_of_two_closed_form(oracle):
    # range = 2^k: value = lo + top k bits of R, R = (w1:w0) for even i, (w3:w2) for odd i
    n = 2048
    for lo, k in [(0, 1), (-(1 << 20), 21), (-(2 ** 31), 32), (100, 7)]:
        v = oracle.synth(1, 1, "i32", "int_range", oracle.dist_params(lo=lo, hi=lo + 2 ** k - 1), n)
        v = v.view(np.int32).astype(np.int64)
        w = oracle.philox_blocks(1, 1, 0, n // 2).astype(np.uint64)
        R = np.empty(n, dtype=np.uint64)
        R[0::2] = (w[:, 1] << np.uint64(32)) | w[:, 0]
        R[1::2] = (w[:, 3] << np.uint64(32)) | w[:, 2]
        want = lo + (R >> np.uint64(64 - k)).astype(np.int64)
        assert np.array_equal(v, want)


def test_int_range_general_is_floor_of_exact_product(oracle):
    lo, hi = -(1 << 20), 1 << 20            # 2^21 + 1 values, inclusive
    n = 4096
    v = oracle.synth(0, 3, "i32", "int_range", oracle.dist_params(lo=lo, hi=hi), n).view(np.int32)
    w = oracle.philox_blocks(0, 3, 0, n // 2)
    for i in range(n):
        h = i % 2
        R = (int(w[i // 2, 2 * h + 1]) << 32) | int(w[i // 2, 2 * h])
        assert int(v[i]) == lo + (R * (hi - lo + 1)) // 2 ** 64


def test_int_range_bounds_endpoints_and_chi_square(oracle):
    v = oracle.synth(0, 0, "i32", "int_range", oracle.dist_params(lo=-3, hi=6), 1 << 20).view(np.int32)
    assert v.min() == -3 and v.max() == 6
    counts = np.bincount(v + 3, minlength=10)
    assert st.chisquare(counts).pvalue > 1e-4
    big = oracle.synth(0, 1, "i32", "int_range", oracle.dist_params(lo=-(1 << 20), hi=1 << 20),
                       1 << 20).view(np.int32)
    assert big.min() >= -(1 << 20) and big.max() <= (1 << 20)
    one = oracle.synth(0, 1, "i32", "int_range", oracle.dist_params(lo=42, hi=42), 100).view(np.int32)
    assert np.all(one == 42)


# --------------------------------------------------------------- special values
SPECIAL = dict(mean=0.0, std=1e3, p_nan=0.01, p_inf=0.005, p_denorm=0.01, p_zero=0.01)


FIB = 0x9E3779B9   # Fibonacci hashing multiplier: 2^32 / golden ratio, odd


def _special_layout(oracle, seed, stream, n, probs):
    """Class of every element as the reading defines it, from the Philox words:
    a candidate when the low byte of its normal word is below S = ceil(256 p),
    then its class word against widths floor(p_class 2^32 256 / S) (exact
    rationals), 0 NaN, 1 Inf, 2 denormal, 3 zero, 4 normal; and the hashed word
    that gives the sign and payload."""
    S = math.ceil(Fraction(256) * sum(Fraction(p) for p in probs))
    w = oracle.philox_blocks(seed, stream, 0, n // 4).reshape(-1)
    q = oracle.philox_blocks(seed, stream, 1 << 62, n // 4).reshape(-1)
    widths = [math.floor(Fraction(p) * 2 ** 40 / S) for p in probs]
    t = np.cumsum(widths)
    cls = np.where((w & 0xFF) < S, np.searchsorted(t, q.astype(np.int64), side="right"), 4)
    cls = np.minimum(cls, 4)
    r = (q.astype(np.uint64) * FIB) & 0xFFFFFFFF
    return S, widths, cls, r.astype(np.uint32)


def test_special_classes_follow_gate_thresholds_and_bit_rules(oracle):
    """Element i = 4c + k: a candidate when the low byte of word k of normal
    block c (bits Box-Muller leaves unused) is below S = ceil(256 p); its class
    from word k of block 2^62 + c; sign and payload / mantissa from that word
    times 0x9E3779B9 mod 2^32; every other element keeps element i of the
    normal distribution with the same (seed, stream, mean, std)."""
    n = 1 << 16
    bits = oracle.synth(0, 0, "f32", "special", oracle.dist_params(**SPECIAL), n)
    S, widths, cls, r = _special_layout(oracle, 0, 0, n, (0.01, 0.005, 0.01, 0.01))
    assert S == 9 and widths == [1221679586, 610839793, 1221679586, 1221679586]
    sign = r & 0x80000000
    mag = bits & 0x7FFFFFFF
    spec = cls < 4
    assert np.all((bits[spec] & 0x80000000) == sign[spec])
    nan = cls == 0
    assert np.all(bits[nan] == (sign[nan] | 0x7FC00000 | (r[nan] & 0x3FFFFF)))
    inf = cls == 1
    assert np.all(mag[inf] == 0x7F800000)
    den = cls == 2
    m = r[den] & 0x7FFFFF
    assert np.all(mag[den] == np.where(m == 0, 1, m))
    assert np.all(mag[cls == 3] == 0)
    nor = cls == 4
    normal = oracle.synth(0, 0, "f32", "normal", oracle.dist_params(mean=0.0, std=1e3), n)
    assert np.array_equal(bits[nor], normal[nor])
    w = oracle.philox_blocks(0, 0, 0, n // 4)
    for i in np.nonzero(nor)[0][:2000]:
        c, k = divmod(int(i), 4)
        zc, zs = oracle.box_muller_f32(int(w[c, 2 * (k // 2)]), int(w[c, 2 * (k // 2) + 1]))
        z = zc if k % 2 == 0 else zs
        assert float(f32(bits[i])) == rne32_exact(Fraction(float(np.float32(1e3))) * Fraction(float(z)))
    x = f32(bits)
    assert np.all(np.isnan(x[nan])) and np.all(np.isinf(x[inf]))
    assert np.all(np.isfinite(x[cls >= 2]))
    assert np.all(np.abs(x[den]) < np.finfo(np.float32).tiny) and np.all(x[den] != 0)


def test_special_class_probabilities_are_the_given_ones(oracle):
    """The share of each class is (S / 256) floor(p 2^32 256 / S) / 2^32: p
    itself, short by less than 2^-32 (exact rationals); and the extremes: no
    special classes gives the normal distribution bit for bit, probabilities
    summing to 1 leave no normal element."""
    for probs in ((0.01, 0.005, 0.01, 0.01), (0.2, 0.1, 0.2, 0.2), (0.25, 0.25, 0.25, 0.25), (1e-6, 0.0, 0.0, 0.3)):
        S = math.ceil(Fraction(256) * sum(Fraction(p) for p in probs))
        for p in probs:
            share = Fraction(S, 256) * math.floor(Fraction(p) * 2 ** 40 / S) / 2 ** 32
            assert 0 <= Fraction(p) - share < Fraction(1, 2 ** 32)
    n = 1 << 14
    none = oracle.synth(3, 1, "f32", "special", oracle.dist_params(mean=5.0, std=10.0), n)
    assert np.array_equal(none, oracle.synth(3, 1, "f32", "normal", oracle.dist_params(mean=5.0, std=10.0), n))
    allp = dict(mean=5.0, std=10.0, p_nan=0.25, p_inf=0.25, p_denorm=0.25, p_zero=0.25)
    x = f32(oracle.synth(3, 1, "f32", "special", oracle.dist_params(**allp), n))
    ax = np.abs(x)
    assert np.all(np.isnan(x) | np.isinf(x) | (ax < np.finfo(np.float32).tiny))
    for cnt in (np.isnan(x).sum(), np.isinf(x).sum(), ((ax > 0) & (ax < np.finfo(np.float32).tiny)).sum(),
                (x == 0).sum()):
        assert abs(cnt - n / 4) < 5 * math.sqrt(n * 3 / 16)


def test_special_signs_payloads_and_independence(oracle):
    """Signs are balanced in every class, each NaN payload bit and the top
    denormal mantissa bits are uniform, and whether an element is special does
    not depend on the normal value it replaces (the normal values at special
    positions follow N(mean, std), KS)."""
    n = 1 << 21
    heavy = dict(mean=0.0, std=1.0, p_nan=0.05, p_inf=0.05, p_denorm=0.05, p_zero=0.05)
    bits = oracle.synth(2, 8, "f32", "special", oracle.dist_params(**heavy), n)
    x = f32(bits)
    ax = np.abs(x)
    tiny = np.finfo(np.float32).tiny
    classes = [np.isnan(x), np.isinf(x), (ax > 0) & (ax < tiny), x == 0]
    for c in classes:
        k = int(c.sum())
        neg = int((bits[c] >> 31).sum())
        assert abs(neg - k / 2) < 5 * math.sqrt(k / 4)
    nanp = bits[classes[0]] & 0x3FFFFF
    for b in range(22):
        ones = int(((nanp >> b) & 1).sum())
        assert abs(ones - nanp.size / 2) < 5 * math.sqrt(nanp.size / 4), b
    top = (bits[classes[2]] & 0x7FFFFF) >> 19                  # top 4 mantissa bits of denormals
    cnt = np.bincount(top, minlength=16)
    e = top.size / 16
    assert ((cnt - e) ** 2 / e).sum() < 15 + 5 * math.sqrt(30)
    spec = ~np.isfinite(x) | (ax < tiny)
    z = f32(oracle.synth(2, 8, "f32", "normal", oracle.dist_params(mean=0.0, std=1.0), n))[spec].astype(np.float64)
    assert st.kstest(z, "norm").statistic < 1.95 / math.sqrt(z.size)


def test_special_class_frequencies(oracle):
    n = 1 << 20
    x = f32(oracle.synth(0, 0, "f32", "special", oracle.dist_params(**SPECIAL), n))
    ax = np.abs(x)
    got = [np.isnan(x).sum(), np.isinf(x).sum(),
           ((ax > 0) & (ax < np.finfo(np.float32).tiny)).sum(), (x == 0).sum()]
    for cnt, p in zip(got, (0.01, 0.005, 0.01, 0.01)):
        assert abs(cnt - n * p) < 5 * math.sqrt(n * p * (1 - p))
    normal = x[np.isfinite(x) & (ax >= np.finfo(np.float32).tiny)].astype(np.float64) / 1e3
    assert st.kstest(normal, "norm").statistic < 1.95 / math.sqrt(normal.size)


# --------------------------------------------------------------- bf16 rounding
def test_bf16_rne_matches_torch(oracle):
    import torch
    rng = np.random.default_rng(0)
    edge = np.array([0, 0x80000000, 1, 0x80000001, 0x007FFFFF, 0x00800000, 0x7F7FFFFF, 0xFF7FFFFF,
                     0x7F800000, 0xFF800000, 0x3F808000, 0x3F818000, 0x3F807FFF, 0x3F808001,
                     0x7F7F8000, 0x7F7F7FFF, 0x00008000, 0x00018000], dtype=np.uint32)
    bits = np.concatenate([edge, rng.integers(0, 2 ** 32, 1 << 20, dtype=np.uint64).astype(np.uint32)])
    finite = (bits & 0x7FFFFFFF) <= 0x7F800000
    got = oracle.bf16_rne_n(bits)
    want = torch.from_numpy(bits.view(np.float32).copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got[finite], want[finite])
    nanb = bits[~finite]
    assert np.all(got[~finite] == ((nanb >> 16) | 0x40).astype(np.uint16))


def test_special_class_counts_agree_with_synthesized_classes(oracle):
    n = 1 << 18
    p = oracle.dist_params(**SPECIAL)
    c = oracle.special_class_counts(0, 5, p, n)
    x = f32(oracle.synth(0, 5, "f32", "special", p, n))
    ax = np.abs(x)
    tiny = np.finfo(np.float32).tiny
    assert list(c) == [np.isnan(x).sum(), np.isinf(x).sum(), ((ax > 0) & (ax < tiny)).sum(),
                       (x == 0).sum(), (np.isfinite(x) & (ax >= tiny)).sum()]
    half = oracle.special_class_counts(0, 5, p, n // 2) + oracle.special_class_counts(0, 5, p, n // 2, offset=n // 2)
    assert np.array_equal(half, c)

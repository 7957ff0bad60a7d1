"""GPU parity of the fp64 check's maxima and error sum where fp64 leaves the
normal range: subnormal references whose quotients d / |y| sit just above a
lane's running maximum, differences of finite values that overflow, and sums
that overflow (Eq. (1) and the report fields of Sec. 4.2.1, read as max over
finite pairs and the fp64 sum of |a - y|).

The check divides d by |y| only where the quotient may beat the lane's running
maximum m, a filter d > fp64(m (1 - 2^-50)) |y|.  Inputs here are built so
that the filter's product is subnormal (or overflows) exactly where a
quotient rounds above m; a filter that trusted the product there would report
a smaller maximum than the oracle.  Each construction is checked on the CPU
to be such a case before it goes to the GPU (regression test of that
filter)."""
import math
import random
from fractions import Fraction

import numpy as np
import pytest
import torch

import paper_2609_00058_amd as sv
from gpu_run import dev_bits, same_report

pytestmark = pytest.mark.gpu

TINY = 2.0 ** -1074          # smallest subnormal: every subnormal is a multiple of it
M_BASE = 0.8294046819550177  # running maximum every lane reaches first
MRC = M_BASE * (1.0 - 2.0 ** -50)   # the filter's factor, rounded as the kernel rounds it


def base_pair():
    """y = 1, a = 1 - m: d = m exactly (Sterbenz), so d / |y| = m."""
    y, a = 1.0, 1.0 - M_BASE
    assert abs(a - y) == M_BASE
    return y, a


def probe_pool(count, seed):
    """Subnormal pairs (y, a) with fp64(d / |y|) > m although d <= fp64(mrc |y|):
    the product rounds up to the candidate's difference.  y = +-k 2^-1074 and
    d = ceil(m k) 2^-1074 with the fractional part of m k at least 1/2."""
    rng = random.Random(seed)
    mf = Fraction(M_BASE)
    out = []
    while len(out) < count:
        k = rng.randrange(1 << 10, 1 << 40)
        mk = mf * k
        if mk - math.floor(mk) < Fraction(1, 2) + Fraction(1, 1 << 20):
            continue
        du = math.ceil(mk)
        y = math.ldexp(k, -1074) * (1 if rng.random() < 0.5 else -1)
        a = y + math.copysign(math.ldexp(du, -1074), y) * (1 if rng.random() < 0.5 else -1)
        d = abs(a - y)
        assert d == math.ldexp(du, -1074)                  # subnormal arithmetic is exact
        q = float(Fraction(du, k))                          # correctly rounded d / |y|
        assert q == d / abs(y) and q > M_BASE
        assert not d > MRC * abs(y)                         # the product-only filter would skip it
        out.append((y, a))
    return out


def layout(n, period_units, pool, nan_lane0=False):
    """fp64 tensors of n elements: within every `period_units` 16-byte units,
    the first half holds base pairs, the second half probes from the pool;
    with nan_lane0, element 0 of every 64th unit is NaN on both sides (so
    every wave takes the non-finite path of the check)."""
    y = np.empty(n, np.float64)
    a = np.empty(n, np.float64)
    by, ba = base_pair()
    unit = np.arange(n) // 2
    probe = (unit % period_units) >= period_units // 2
    y[~probe], a[~probe] = by, ba
    py = np.array([p[0] for p in pool]), np.array([p[1] for p in pool])
    pi = np.nonzero(probe)[0]
    sel = np.arange(pi.size) % len(pool)
    y[pi], a[pi] = py[0][sel], py[1][sel]
    if nan_lane0:
        z = np.nonzero((unit % 64 == 0) & (np.arange(n) % 2 == 0))[0]
        y[z] = np.nan
        a[z] = np.nan
    return y, a


def run_both(oracle, y, a, rtol=1e-7, atol=0.0, equal_nan=True):
    yb, ab = y.view(np.uint64), a.view(np.uint64)
    want = oracle.compare(yb, ab, "f64", rtol, atol, equal_nan)
    ref, cand = dev_bits(yb, "f64"), dev_bits(ab, "f64")
    got = sv.compare(ref, cand, rtol, atol, equal_nan)
    same_report(got, want)
    [bat] = sv.compare_batched([(ref, cand, rtol, atol, equal_nan)])
    same_report(bat, want)
    return got, want


@pytest.mark.parametrize("nan_lane0", [False, True])
def test_subnormal_quotients_just_above_the_running_maximum(oracle, nan_lane0):
    pool = probe_pool(512, seed=11)
    best = max(abs(a - y) / abs(y) for y, a in pool)
    # one workgroup: every lane checks its units of the base half (units < 2048)
    # before those of the probe half, so each probe meets the maximum m
    print("fp64 near ties, one workgroup, nan_lane0 =", nan_lane0, flush=True)
    y, a = layout(8192, 4096, pool, nan_lane0)
    got, want = run_both(oracle, y, a)
    assert want["max_rel_err"] == best > M_BASE
    # many workgroups: chunks of whole 1024-unit periods; in each tile a lane
    # meets a base unit, then a probe unit, twice
    print("fp64 near ties, 2^25 elements, nan_lane0 =", nan_lane0, flush=True)
    y, a = layout(1 << 25, 1024, pool, nan_lane0)
    got, want = run_both(oracle, y, a)
    assert want["max_rel_err"] == best
    del y, a
    torch.cuda.empty_cache()


def test_overflowing_differences_and_sums(oracle):
    """d = |a - y| of two finite values may overflow to +Inf (then d, max abs,
    max rel and the sum are +Inf), and finite differences may sum past the
    largest fp64 value (the sum is +Inf, never NaN)."""
    print("fp64 overflow: infinite difference after a finite maximum", flush=True)
    n = 8192
    y = np.ones(n)
    a = -np.ones(n)                                  # d = 2, d / |y| = 2 everywhere in the first half
    probes = np.arange(4096, n, 97)
    y[probes], a[probes] = 1e308, -1e308             # d overflows: quotient +Inf
    got, want = run_both(oracle, y, a, rtol=1.0, atol=0.0, equal_nan=False)
    assert want["max_rel_err"] == math.inf and want["max_abs_err"] == math.inf and want["err_sum"] == math.inf
    print("fp64 overflow: finite differences whose sum overflows", flush=True)
    for n in (2, 4097, 1 << 20):
        y = np.full(n, 1e308)
        a = np.full(n, -7e307)                       # d = 1.7e308 each, finite
        got, want = run_both(oracle, y, a, rtol=1.0, atol=0.0, equal_nan=False)
        assert want["err_sum"] == math.inf and want["max_abs_err"] == 1.7e308
    print("fp64 overflow: large but finite sum", flush=True)
    y = np.zeros(1000)
    a = np.full(1000, 1e305)
    got, want = run_both(oracle, y, a, rtol=1.0, atol=0.0, equal_nan=False)
    assert math.isfinite(want["err_sum"])

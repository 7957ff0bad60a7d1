"""Seeded random batches through every check entry point, against the oracle.

Thirty batches of up to thirteen segments each: every element type, lengths
from empty to a few hundred thousand elements, views that start one to three
elements into their buffers (the element path), candidates equal to their
reference, aliased to it, or differing with special values mixed in, and
random tolerances and equal_nan.  Each batch goes through the plain batched
check, the stop-at-first check, a submitted check waited for later, and two of
its segments through the single-tensor check and the check without
allocation.  Reports must equal the oracle's (the fp64 error sum within 1e-12
relative); a failing segment of a stop-at-first check carries the exact first
index.
"""
import numpy as np
import pytest

import paper_2609_00058_amd as sv
from gpu_run import STORAGE, dev_bits, same_report

pytestmark = pytest.mark.gpu

TYPES = ["f32", "bf16", "i32", "f16", "f64", "u8", "i64"]


def _values(rng, n, dtype):
    from test_gpu_compare import random_pair
    from test_gpu_dtypes import _pair
    if n == 0:
        return np.empty(0, STORAGE[dtype]), np.empty(0, STORAGE[dtype])
    if dtype in ("f32", "bf16", "i32"):
        return random_pair(rng, n, dtype, special_frac=float(rng.choice([0.0, 0.01, 0.2])))
    return _pair(rng, n, dtype)


def _length(rng):
    r = rng.random()
    if r < 0.1:
        return 0
    if r < 0.4:
        return int(rng.integers(1, 65))
    if r < 0.8:
        return int(rng.integers(65, 5000))
    return int(rng.integers(5000, 200000))


def _tolerance(rng):
    rtol = 0.0 if rng.random() < 0.2 else float(10.0 ** rng.uniform(-9, 0))
    atol = 0.0 if rng.random() < 0.3 else float(10.0 ** rng.uniform(-45, 0))
    return rtol, atol, bool(rng.integers(0, 2))


@pytest.mark.parametrize("seed", range(30))
def test_random_batches_match_the_oracle(oracle, seed):
    rng = np.random.default_rng(9000 + seed)
    segs, want, keep = [], [], []
    for k in range(int(rng.integers(1, 14))):
        dtype = TYPES[int(rng.integers(0, len(TYPES)))]
        n, off = _length(rng), int(rng.integers(0, 4))
        y, a = _values(rng, n + off, dtype)
        kind = rng.random()
        if kind < 0.2:
            a = y.copy()                         # a candidate that passes
        Y = dev_bits(y, dtype)
        A = Y if kind > 0.9 else dev_bits(a, dtype)   # aliased: the reference checked against itself
        if kind > 0.9:
            a = y
        keep += [Y, A]
        rtol, atol, eqn = _tolerance(rng)
        segs.append((Y[off:off + n], A[off:off + n], rtol, atol, eqn))
        want.append(oracle.compare(y[off:off + n], a[off:off + n], dtype, rtol, atol, eqn))
    print("fuzz batch", seed, [(s[0].dtype, s[0].numel()) for s in segs], flush=True)

    for g, w in zip(sv.compare_batched(segs), want):
        same_report(g, w)
    for g, w in zip(sv.compare_batched(segs, stop_at_first=True), want):
        if w["mismatches"] == 0:
            same_report(g, w)
        else:
            assert g["mismatches"] == 1 and g["first_mismatch"] == w["first_mismatch"], (g, w)
    stop = bool(rng.integers(0, 2))
    ticket = sv.compare_batched_submit(segs, stop_at_first=stop)
    for g, w in zip(ticket.wait(), want):
        if not stop or w["mismatches"] == 0:
            same_report(g, w)
        else:
            assert g["first_mismatch"] == w["first_mismatch"]
    for j in rng.choice(len(segs), size=min(2, len(segs)), replace=False):
        same_report(sv.compare(*segs[int(j)]), want[int(j)])
        same_report(sv.compare_noalloc(*segs[int(j)]), want[int(j)])


def test_twenty_thousand_small_segments(oracle):
    """A batch far longer than the grid: 20,000 segments of 0 to 50 elements
    of every type, in one buffer per type, both check modes."""
    rng = np.random.default_rng(9100)
    pools = {}
    for dtype in TYPES:
        y, a = _values(rng, 600_000, dtype)
        pools[dtype] = (y, a, dev_bits(y, dtype), dev_bits(a, dtype))
    segs, want = [], []
    for k in range(20000):
        dtype = TYPES[k % len(TYPES)]
        y, a, Y, A = pools[dtype]
        n = int(rng.integers(0, 51))
        o = int(rng.integers(0, 600_000 - n))
        rtol, atol, eqn = _tolerance(rng)
        segs.append((Y[o:o + n], A[o:o + n], rtol, atol, eqn))
        want.append(oracle.compare(y[o:o + n], a[o:o + n], dtype, rtol, atol, eqn))
    print("twenty thousand segments", flush=True)
    got = sv.compare_batched(segs)
    for g, w in zip(got, want):
        same_report(g, w)
    for g, w in zip(sv.compare_batched(segs, stop_at_first=True), want):
        if w["mismatches"] == 0:
            same_report(g, w)
        else:
            assert g["mismatches"] == 1 and g["first_mismatch"] == w["first_mismatch"], (g, w)


TOL_EXTREMES = [(0.0, 0.0), (1e308, 0.0), (0.0, 1e308), (1.7976931348623157e308, 1.7976931348623157e308),
                (5e-324, 5e-324), (-0.0, -0.0), (-1e-9, 0.0), (0.0, -1e-9), (float("nan"), 0.0),
                (0.0, float("nan")), (float("inf"), 0.0), (0.0, float("inf"))]


@pytest.mark.parametrize("rtol,atol", TOL_EXTREMES)
@pytest.mark.parametrize("dtype", ["f32", "f64", "i32"])
def test_extreme_tolerances_agree_with_the_oracle(oracle, dtype, rtol, atol):
    """Tolerances at the ends of fp64 and outside the allowed range: refused by
    the library exactly where the oracle refuses them, otherwise the oracle's
    report (single and batched)."""
    rng = np.random.default_rng(9600)
    y, a = _values(rng, 3001, dtype)
    try:
        want = oracle.compare(y, a, dtype, rtol, atol, True)
    except oracle.OracleError:
        want = None
    Y, A = dev_bits(y, dtype), dev_bits(a, dtype)
    for call in (lambda: sv.compare(Y, A, rtol, atol, True),
                 lambda: sv.compare_batched([(Y, A, rtol, atol, True)])[0]):
        try:
            got = call()
        except sv.SVError:
            got = None
        if want is None:
            assert got is None, "the library accepted what the oracle refuses"
        else:
            assert got is not None, "the library refused what the oracle accepts"
            same_report(got, want)

"""The library refuses exactly the arguments the oracle refuses.

Property tests over the parameters of synthesis, candidate steps and the
check: element types and distributions (valid and unknown codes), bounds,
means and widths at the ends of fp32 and fp64 and beyond them, NaN and
infinite values, probabilities outside [0, 1] and sums just above 1, integer
ranges at and past the limits of each type, permutation domains and windows,
selection probabilities, widths, deltas, index lists, and tolerances.  For
every drawn case the oracle's status decides: where it refuses, the library
must return SV_ERR_INVALID_ARG or SV_ERR_UNSUPPORTED; where it accepts, the
library must pass its argument checks and reach the device, which this
container does not have (SV_ERR_HIP).  The library's pointers are stand-ins
that no device ever sees, so the test runs only where there is no GPU.

Two limits are the library's own and are checked apart from the oracle: a
window ends at or below 2^60 elements, and an index list names elements of
the tensor (the oracle's windows skip indices outside them).
"""
import ctypes
import math
import os

import numpy as np
import pytest
from hypothesis import HealthCheck, event, given, settings, strategies as st

import oracle

pytestmark = pytest.mark.skipif(os.path.exists("/dev/kfd"),
                                reason="stand-in device pointers are only safe where there is no GPU")

SETTINGS = settings(max_examples=1500, derandomize=True, deadline=None,
                    suppress_health_check=[HealthCheck.too_slow])

F32_MAX = float(np.finfo(np.float32).max)
EDGE = [0.0, 1.0, 0.5, 1.5, 2.0, 1e-3, 0.1, 1e-7, 1e3, 1e-45, 1.401298464324817e-45, 1.1754943508222875e-38,
        5e-324, 2.2250738585072014e-308, 65504.0, 65520.0, F32_MAX, 3.4028235677973366e38, 3.5e38, 1e300,
        1.7976931348623157e308, math.inf, math.nan, 1.0 - 2.0 ** -53, 1.0 + 2.0 ** -52, 1.0 - 2.0 ** -24]
EDGE = EDGE + [-x for x in EDGE]
I64 = (-2 ** 63, 2 ** 63 - 1)
INT_EDGE = [0, 1, -1, 2, 9, 100, 255, 256, -2 ** 31 - 1, -2 ** 31, 2 ** 31 - 1, 2 ** 31, 2 ** 32, 2 ** 60 - 1,
            2 ** 60, 2 ** 60 + 1, -2 ** 60, I64[0], I64[0] + 1, I64[1] - 1, I64[1]]
OFFSET_EDGE = [0, 1, 3, 95, 2 ** 32, 2 ** 40, 2 ** 60 - 16, 2 ** 60 - 1, 2 ** 60]

real = st.one_of(st.sampled_from(EDGE), st.floats(allow_nan=True, allow_infinity=True),
                 st.floats(-4.0, 4.0))
prob = st.one_of(st.sampled_from([0.0, 1.0, 0.5, 0.25, 0.2, 1.0 + 2.0 ** -52, 1e-300, -0.0, -1e-300, 0.6, math.nan,
                                  math.inf, 1.0 / 3.0]), st.floats(-0.5, 1.5))
whole = st.one_of(st.sampled_from(INT_EDGE), st.integers(*I64), st.integers(-300, 300))
dtype = st.sampled_from(list(range(7)) * 3 + [-1, 7, 100])
length = st.sampled_from([0, 1, 2, 3, 4, 5, 8, 16, 17, 64])


def _rc(svlib, rc):
    """'refused', 'accepted' (the argument checks passed: the call reached for
    the device, or had nothing to do), or the unexpected status itself."""
    if rc in (svlib.SV_ERR_INVALID_ARG, svlib.SV_ERR_UNSUPPORTED):
        return "refused"
    return "accepted" if rc in (svlib.SV_ERR_HIP, svlib.SV_OK) else rc


@pytest.fixture(scope="module")
def svlib():
    import paper_2609_00058_amd as sv
    return sv


VALID_TYPES = {0: [0, 1, 3, 4], 1: [0, 1, 3, 4], 3: [0, 1, 3, 4], 2: [2, 5, 6], 4: [2, 5, 6]}
TYPE_RANGE = {2: (-2 ** 31, 2 ** 31 - 1), 5: (0, 255), 6: I64}
SUMS_TO_ONE = [(1.0, 0.0, 0.0, 0.0), (0.5, 0.5, 0.0, 0.0), (0.25, 0.25, 0.25, 0.25), (0.5, 0.25, 0.125, 0.125),
               (0.5, 0.25, 0.125, 0.125 + 2.0 ** -52), (0.6, 0.4, 0.0, 0.0), (0.1, 0.2, 0.3, 0.4),
               (1.0 - 2.0 ** -53, 2.0 ** -53, 0.0, 0.0), (1.0, 5e-324, 0.0, 0.0), (0.7, 0.2, 0.1, 0.0)]


def _params(draw, dist, dt):
    """Half of the draws well-formed for the pair (valid values, perhaps at the
    edges), half from the edge sets (mostly refused)."""
    tame = draw(st.booleans())
    if dist == 0:
        a = draw(st.floats(-1e30, 1e30) if tame else real)
        width = st.floats(1e-30, 1e30) if tame else real
        b = draw(st.one_of(st.builds(lambda d: a + abs(d), width), real,
                           st.just(float(np.nextafter(np.float32(a), np.float32(math.inf))))
                           if math.isfinite(a) and abs(a) <= F32_MAX else real))
        return dict(a=a, b=b)
    if dist in (1, 3):
        kw = dict(mean=draw(st.floats(-1e30, 1e30) if tame else real),
                  std=draw(st.floats(0.0, 1e30) if tame else real))
        if dist == 3:
            if tame and draw(st.booleans()):
                ps = list(draw(st.permutations(draw(st.sampled_from(SUMS_TO_ONE)))))
            elif tame:
                w = draw(st.lists(st.floats(0.0, 1.0), min_size=5, max_size=5))
                tot = sum(w) or 1.0
                ps = [x / tot * draw(st.floats(0.0, 1.0)) for x in w[:4]]
            else:
                ps = [draw(prob) for _ in range(4)]
            kw.update(p_nan=ps[0], p_inf=ps[1], p_denorm=ps[2], p_zero=ps[3])
        return kw
    if dist in (2, 4):
        lo_t, hi_t = TYPE_RANGE.get(dt, I64)
        lo = draw(st.integers(lo_t, hi_t) if tame else whole)
        near = [max(I64[0], min(I64[1], v)) for v in (hi_t, hi_t + 1, lo_t, lo_t - 1, lo, lo - 1, lo + 1)]
        hi = draw(st.one_of(whole, st.integers(lo_t, hi_t), st.sampled_from(near),
                            st.builds(lambda d: max(I64[0], min(I64[1], lo + d)), st.integers(-2, 2 ** 20))))
        return dict(lo=lo, hi=hi)
    return dict(a=draw(real), b=draw(real), mean=draw(real), std=draw(real), lo=draw(whole), hi=draw(whole))


@st.composite
def synth_case(draw):
    dist = draw(st.sampled_from([0, 1, 2, 3, 4] * 4 + [-1, 5]))
    if dist in VALID_TYPES and draw(st.integers(0, 4)):
        dt = draw(st.sampled_from(VALID_TYPES[dist]))
    else:
        dt = draw(dtype)
    return dict(dtype=dt, dist=dist, kw=_params(draw, dist, dt), n=draw(length),
                offset=draw(st.one_of(st.sampled_from(OFFSET_EDGE), st.integers(0, 2 ** 60))))


def _oracle_synth(c, offset):
    p = oracle.dist_params(**c["kw"])
    out = np.empty(c["n"], np.uint64)
    rc = oracle.lib().or_synth(3, 4, c["dtype"], c["dist"], ctypes.byref(p), offset, c["n"],
                               out.ctypes.data_as(ctypes.c_void_p))
    return "refused" if rc else "accepted"


@SETTINGS
@given(synth_case())
def test_synthesis_parameters(svlib, c):
    L = svlib.lib()
    p = svlib.dist_params(**c["kw"])
    want = _oracle_synth(c, 0)
    event("synthesis %s" % want)
    assert _rc(svlib, L.sv_synth(3, 4, c["dtype"], c["dist"], ctypes.byref(p), c["n"], 0x10000)) == want, c
    job = svlib.SynthJob(3, 4, c["dtype"], c["dist"], p, c["n"], 0x10000)
    assert _rc(svlib, L.sv_synth_batched(ctypes.byref(job), 1)) == want, c
    off = c["offset"]
    rc = _rc(svlib, L.sv_synth_window(3, 4, c["dtype"], c["dist"], ctypes.byref(p), off, c["n"], 0x10000))
    if off + c["n"] > 2 ** 60:
        assert rc == "refused", c                       # the library's own limit on windows
    else:
        assert rc == _oracle_synth(c, off), c


@st.composite
def perturb_case(draw):
    n = draw(length)
    op = draw(st.one_of(st.integers(0, 6), st.sampled_from([-1, 7])))
    idx = draw(st.lists(st.one_of(st.integers(0, max(n - 1, 0)), st.sampled_from([n, n + 1, 2 ** 64 - 1])),
                        max_size=6))
    return dict(dtype=draw(dtype), op=op, n=n, p=draw(prob), value=draw(real),
                bits=draw(st.integers(0, 2 ** 32 - 1)), idx=idx)


@SETTINGS
@given(perturb_case())
def test_candidate_step_parameters(svlib, c):
    L = svlib.lib()
    idx = np.array(c["idx"], dtype=np.uint64)
    ptr = idx.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64))
    plan = oracle.PerturbPlan(c["op"], c["p"], c["value"], c["bits"], ptr, idx.size)
    ref = np.zeros(c["n"], np.uint64)
    cand = np.zeros(c["n"], np.uint64)
    rc = oracle.lib().or_perturb(5, 6, c["dtype"], ctypes.byref(plan), 0, c["n"],
                                 ref.ctypes.data_as(ctypes.c_void_p), cand.ctypes.data_as(ctypes.c_void_p))
    want = "refused" if rc else "accepted"
    event("step %s" % want)
    splan = svlib.PerturbPlan(c["op"], c["p"], c["value"], c["bits"], ptr, idx.size)
    got = _rc(svlib, L.sv_perturb(5, 6, c["dtype"], ctypes.byref(splan), c["n"], 0x10000, 0x20000))
    if c["op"] in (4, 5, 6) and want == "accepted" and (idx >= c["n"]).any():
        assert got == "refused", c                      # the library's indices name elements of the tensor
    else:
        assert got == want, c


tol = st.one_of(st.sampled_from([0.0, -0.0, 1e-5, 1e-8, 5e-324, 1e308, 1.7976931348623157e308, math.inf,
                                 -math.inf, math.nan, -1e-9]), st.floats(allow_nan=True, allow_infinity=True))


@SETTINGS
@given(dtype, tol, tol, st.booleans(), length)
def test_check_tolerances(svlib, dt, rtol, atol, eqn, n):
    L = svlib.lib()
    ref = np.zeros(n, np.uint64)
    r = oracle.Report()
    rc = oracle.lib().or_compare(ref.ctypes.data_as(ctypes.c_void_p), ref.ctypes.data_as(ctypes.c_void_p), n, dt,
                                 rtol, atol, int(eqn), ctypes.byref(r))
    want = "refused" if rc else "accepted"
    event("check %s" % want)
    rep = svlib.Report()
    reps = (svlib.Report * 1)()
    ticket = ctypes.c_uint64(0)
    seg = (svlib.Segment * 1)(svlib.Segment(0x10000, 0x20000, n, dt, rtol, atol, int(eqn)))
    calls = {
        "compare": lambda: L.sv_compare(0x10000, 0x20000, n, dt, rtol, atol, int(eqn), ctypes.byref(rep)),
        "noalloc": lambda: L.sv_compare_noalloc(0x10000, 0x20000, n, dt, rtol, atol, int(eqn), ctypes.byref(rep)),
        "submit": lambda: L.sv_compare_submit(0x10000, 0x20000, n, dt, rtol, atol, int(eqn), ctypes.byref(ticket)),
        "batched": lambda: L.sv_compare_batched(seg, 1, reps),
        "stop_at_first": lambda: L.sv_compare_batched_mode(seg, 1, 1, reps),
        "batched_submit": lambda: L.sv_compare_batched_submit(seg, 1, 0, ctypes.byref(ticket)),
    }
    for name, call in calls.items():
        assert _rc(svlib, call()) == want, (name, dt, rtol, atol, eqn, n)


def _edges_int(dt):
    lo_t, hi_t = TYPE_RANGE[dt]
    vals = {lo_t - 1, lo_t, lo_t + 1, -1, 0, 1, 255, 256, hi_t - 1, hi_t, hi_t + 1, 2 ** 60 - 1, 2 ** 60,
            lo_t + 2 ** 60 - 1, lo_t + 2 ** 60}
    return sorted(v for v in vals if I64[0] <= v <= I64[1])


F_GRID = [-math.inf, -1.7976931348623157e308, -3.5e38, -3.4028235677973366e38, -F32_MAX, -1.0, -1e-45, -0.0, 0.0,
          5e-324, 1e-45, 1.0, float(np.nextafter(np.float32(1.0), np.float32(2.0))), 65504.0, 65520.0, F32_MAX,
          3.4028235677973366e38, 3.5e38, 1.7976931348623157e308, math.inf, math.nan]


def test_synthesis_parameter_grid(svlib):
    """Every pair of edge values for each distribution and element type (the
    edges a random draw rarely hits together)."""
    L = svlib.lib()
    cases = []
    for dist in (2, 4):
        for dt in (2, 5, 6):
            cases += [dict(dtype=dt, dist=dist, kw=dict(lo=lo, hi=hi), n=1) for lo in _edges_int(dt)
                      for hi in _edges_int(dt)]
    for dt in (0, 1, 3, 4):
        cases += [dict(dtype=dt, dist=0, kw=dict(a=a, b=b), n=4) for a in F_GRID for b in F_GRID]
        cases += [dict(dtype=dt, dist=1, kw=dict(mean=m, std=s), n=4) for m in F_GRID for s in F_GRID]
        ps = SUMS_TO_ONE + [(1.0 + 2.0 ** -52, 0.0, 0.0, 0.0), (-0.0, 0.0, 0.0, 0.0), (math.nan, 0.0, 0.0, 0.0),
                            (0.5, 0.5, 2.0 ** -53, 0.0), (0.0, 0.0, 0.0, -5e-324), (math.inf, 0.0, 0.0, 0.0)]
        cases += [dict(dtype=dt, dist=3, kw=dict(mean=m, std=1.0, p_nan=p[0], p_inf=p[1], p_denorm=p[2],
                                                 p_zero=p[3]), n=4) for m in F_GRID for p in ps]
    counts = {"accepted": 0, "refused": 0}
    for c in cases:
        p = svlib.dist_params(**c["kw"])
        want = _oracle_synth(c, 0)
        counts[want] += 1
        assert _rc(svlib, L.sv_synth(3, 4, c["dtype"], c["dist"], ctypes.byref(p), c["n"], 0x10000)) == want, c
    assert min(counts.values()) > 500, counts


def test_permutation_window_grid(svlib):
    """Windows at, inside and just past the end of small permutation domains,
    empty windows included."""
    L = svlib.lib()
    seen = {"accepted": 0, "refused": 0}
    for dt in (2, 5, 6):
        for r in (1, 2, 10, 100):
            p = svlib.dist_params(lo=7, hi=7 + r - 1)
            for off in (0, 1, r - 1, r, r + 1):
                for n in sorted({0, 1, max(r - off, 0), r - off + 1}):
                    c = dict(dtype=dt, dist=4, kw=dict(lo=7, hi=7 + r - 1), n=n)
                    want = _oracle_synth(c, off)
                    seen[want] += 1
                    got = _rc(svlib, L.sv_synth_window(3, 4, dt, 4, ctypes.byref(p), off, n, 0x10000))
                    assert got == want, (c, off)
    assert min(seen.values()) > 20, seen

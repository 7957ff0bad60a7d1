"""Seeded random synthesis requests through sv_synth, sv_synth_window and
sv_synth_batched, bit for bit against the oracle.

Forty requests, each with a random seed, stream, distribution and element
type, random parameters (bounds and spans from 10^-3 to 10^3, integer ranges
up to the whole type, class probabilities that sum to anything up to 1,
permutation domains from one value to 2^20), lengths from 0 to 70,000,
windows starting anywhere below 2^40, and outputs that start zero to three
elements into their buffers (the element-by-element path); then all of the
whole-tensor requests again as one batch.
"""
import numpy as np
import pytest

import paper_2609_00058_amd as sv
from gpu_run import bits, empty

pytestmark = pytest.mark.gpu

FLOATS = ["f32", "bf16", "f16", "f64"]
INTS = ["i32", "u8", "i64"]
LIMITS = {"i32": (-2 ** 31, 2 ** 31 - 1), "u8": (0, 255), "i64": (-2 ** 63, 2 ** 63 - 1)}


def _request(rng):
    dist = str(rng.choice(["uniform", "normal", "int_range", "special", "permutation"]))
    dtype = str(rng.choice(INTS if dist in ("int_range", "permutation") else FLOATS))
    n = int(rng.choice([0, int(rng.integers(1, 100)), int(rng.integers(100, 70000))]))
    if dist == "uniform":
        a = float(rng.uniform(-1e3, 1e3))
        params = dict(a=a, b=a + float(10.0 ** rng.uniform(-3, 3)))
    elif dist == "normal":
        params = dict(mean=float(rng.uniform(-100, 100)), std=float(10.0 ** rng.uniform(-3, 3)))
    elif dist == "special":
        p = rng.dirichlet(np.ones(5)) * (1.0 if rng.random() < 0.2 else float(rng.uniform(0, 1)))
        params = dict(mean=float(rng.uniform(-100, 100)), std=float(10.0 ** rng.uniform(-3, 3)),
                      p_nan=float(p[0]), p_inf=float(p[1]), p_denorm=float(p[2]), p_zero=float(p[3]))
    else:
        lo_t, hi_t = LIMITS[dtype]
        if dist == "int_range" and rng.random() < 0.2:
            lo, hi = lo_t, hi_t
        else:
            span = int(min(hi_t - lo_t, int(10.0 ** rng.uniform(0, 18 if dtype == "i64" else 9))))
            if dist == "permutation":
                span = min(span, (1 << 20) - 1)
            lo = int(rng.integers(lo_t, hi_t - span + 1)) if hi_t - span > lo_t else lo_t
            hi = lo + span
        params = dict(lo=lo, hi=hi)
        if dist == "permutation":
            n = min(n, hi - lo + 1)
    offset = 0 if rng.random() < 0.5 else int(rng.integers(0, 1 << 40))
    if dist == "permutation":
        offset = 0 if offset == 0 else int(rng.integers(0, params["hi"] - params["lo"] + 1 - n + 1))
    return dict(seed=int(rng.integers(0, 2 ** 63)), stream=int(rng.integers(0, 2 ** 63)), dist=dist,
                dtype=dtype, n=n, params=params, offset=offset, shift=int(rng.integers(0, 4)))


def _want(oracle, r, offset):
    return oracle.synth(r["seed"], r["stream"], r["dtype"], r["dist"], oracle.dist_params(**r["params"]), r["n"],
                        offset=offset)


def test_random_requests_match_the_oracle(oracle):
    rng = np.random.default_rng(9200)
    reqs = [_request(rng) for _ in range(40)]
    batch = []
    for k, r in enumerate(reqs):
        print("synth fuzz", k, r["dist"], r["dtype"], r["n"], r["offset"], r["shift"], flush=True)
        buf = empty(r["n"] + 4, r["dtype"])
        out = buf[r["shift"]:r["shift"] + r["n"]]
        sv.synth_window(out, r["seed"], r["stream"], r["dist"], r["offset"], **r["params"])
        want = _want(oracle, r, r["offset"])
        assert np.array_equal(bits(out), want.view(bits(out).dtype)), (k, r)
        whole = empty(r["n"], r["dtype"])
        sv.synth(whole, r["seed"], r["stream"], r["dist"], **r["params"])
        w0 = _want(oracle, r, 0)
        assert np.array_equal(bits(whole), w0.view(bits(whole).dtype)), (k, r)
        batch.append((empty(r["n"], r["dtype"]), r, w0))
    print("synth fuzz batch", len(batch), flush=True)
    sv.synth_batched([(o, r["seed"], r["stream"], r["dist"], r["params"]) for o, r, _ in batch])
    for k, (o, r, w0) in enumerate(batch):
        assert np.array_equal(bits(o), w0.view(bits(o).dtype)), (k, r)


EXTREME = [("uniform", "f32", dict(a=-3e38, b=3e38)), ("uniform", "f64", dict(a=-1.7e308, b=1.7e308)),
           ("uniform", "bf16", dict(a=1.0, b=1.0)), ("uniform", "f32", dict(a=1.0, b=1.0000001)),
           ("uniform", "f32", dict(a=0.0, b=1e-40)), ("uniform", "f16", dict(a=-1e6, b=1e6)),
           ("uniform", "f64", dict(a=-1e-310, b=1e-310)), ("normal", "f32", dict(mean=0.0, std=1e38)),
           ("normal", "f32", dict(mean=3e38, std=1e38)), ("normal", "bf16", dict(mean=-3e38, std=1e38)),
           ("normal", "f16", dict(mean=0.0, std=1e5)), ("normal", "f64", dict(mean=1e300, std=1e38)),
           ("normal", "f32", dict(mean=0.0, std=0.0)), ("normal", "f32", dict(mean=1e-45, std=1e-45)),
           ("special", "f32", dict(mean=0.0, std=1e38, p_nan=0.25, p_inf=0.25, p_denorm=0.25, p_zero=0.25)),
           ("special", "f16", dict(mean=6e4, std=1e4, p_nan=0.0, p_inf=0.0, p_denorm=0.5, p_zero=0.0)),
           ("int_range", "i32", dict(lo=5, hi=5)), ("int_range", "u8", dict(lo=255, hi=255)),
           ("int_range", "i64", dict(lo=-2 ** 63, hi=-2 ** 63 + 1)), ("permutation", "u8", dict(lo=7, hi=7)),
           ("int_range", "i64", dict(lo=-2 ** 63, hi=2 ** 63 - 1)), ("int_range", "u8", dict(lo=0, hi=255)),
           ("permutation", "u8", dict(lo=0, hi=255)), ("permutation", "i32", dict(lo=-2 ** 31, hi=2 ** 31 - 1)),
           ("permutation", "i64", dict(lo=-2 ** 63, hi=-2 ** 63 + 2 ** 60 - 1)),
           ("permutation", "i64", dict(lo=2 ** 63 - 2 ** 60, hi=2 ** 63 - 1)),
           ("uniform", "f16", dict(a=-65504.0, b=65504.0)), ("uniform", "bf16", dict(a=-3e38, b=3e38)),
           ("normal", "f64", dict(mean=0.0, std=3.4e38)),
           ("special", "bf16", dict(mean=0.0, std=1.0, p_nan=0.0, p_inf=0.0, p_denorm=1.0, p_zero=0.0)),
           ("special", "f64", dict(mean=0.0, std=1.0, p_nan=1.0, p_inf=0.0, p_denorm=0.0, p_zero=0.0))]


@pytest.mark.parametrize("dist,dtype,params", EXTREME)
def test_extreme_parameters_agree_with_the_oracle(oracle, dist, dtype, params):
    """Spans and scales at the ends of the types, whole-type integer ranges and
    permutation domains up to 2^60 values: the library refuses exactly what
    the oracle refuses, and otherwise writes the oracle's bits (values that
    overflow to infinity included)."""
    n = 40_001 if dist != "permutation" else min(40_001, params["hi"] - params["lo"] + 1)
    try:
        want = oracle.synth(3, 4, dtype, dist, oracle.dist_params(**params), n)
    except oracle.OracleError:
        want = None
    out = empty(n, dtype)
    try:
        sv.synth(out, 3, 4, dist, **params)
        got = bits(out)
    except sv.SVError:
        got = None
    if want is None:
        assert got is None, "the library accepted what the oracle refuses"
    else:
        assert got is not None, "the library refused what the oracle accepts"
        assert np.array_equal(got, want.view(got.dtype))

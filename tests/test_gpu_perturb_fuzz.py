"""Seeded random candidate-derivation steps (sv_perturb) against the oracle.

Sixty steps: every element type, every op, random selection probabilities,
scale widths, deltas, bit patterns and index lists (duplicates included),
references of normal, special-value and integer data, lengths from 0 to
50,000, views one to three elements into their buffers, and in place
(cand = ref) as well as into a separate tensor.  Where the oracle refuses a
combination the library must refuse it too; otherwise the candidate's bits
must equal the oracle's.
"""
import numpy as np
import pytest

import paper_2609_00058_amd as sv
from gpu_run import bits, dev_bits, empty

pytestmark = pytest.mark.gpu

TYPES = ["f32", "bf16", "i32", "f16", "f64", "u8", "i64"]
OPS = ["copy", "ulp", "scale", "special_flip", "add_at", "set_at", "fault_at"]
SPECIAL = dict(mean=0.0, std=1e3, p_nan=0.05, p_inf=0.05, p_denorm=0.05, p_zero=0.1)


def _reference(oracle, rng, dtype, n):
    if dtype in ("i32", "u8", "i64"):
        lo, hi = {"i32": (-2 ** 31, 2 ** 31 - 1), "u8": (0, 255), "i64": (-2 ** 63, 2 ** 63 - 1)}[dtype]
        p = oracle.dist_params(lo=lo, hi=hi)
        return oracle.synth(int(rng.integers(0, 2 ** 62)), 1, dtype, "int_range", p, n)
    if rng.random() < 0.5:
        return oracle.synth(int(rng.integers(0, 2 ** 62)), 2, dtype, "special", oracle.dist_params(**SPECIAL), n)
    return oracle.synth(int(rng.integers(0, 2 ** 62)), 3, dtype, "normal", oracle.dist_params(mean=5.0, std=10.0), n)


def test_random_steps_match_the_oracle(oracle):
    rng = np.random.default_rng(9300)
    done = refused = 0
    for k in range(60):
        dtype = TYPES[int(rng.integers(0, len(TYPES)))]
        op = OPS[int(rng.integers(0, len(OPS)))]
        n = int(rng.choice([0, int(rng.integers(1, 64)), int(rng.integers(64, 50000))]))
        shift = int(rng.integers(0, 4))
        seed, stream = int(rng.integers(0, 2 ** 63)), int(rng.integers(0, 2 ** 63))
        kw = dict(p=float(rng.choice([0.0, 1.0, rng.random()])), value=float(rng.choice([1e-3, 0.5, -2.0, 1e30])),
                  bits=int(rng.integers(0, 2 ** 32)))
        idx = None
        if op in ("add_at", "set_at", "fault_at"):
            idx = np.sort(rng.integers(0, n, int(rng.integers(0, 20)))).astype(np.uint64) if n else \
                np.empty(0, np.uint64)
        ref = _reference(oracle, rng, dtype, n)
        try:
            want = oracle.perturb(seed, stream, dtype, op, ref, ref.copy(), idx=idx, **kw)
        except oracle.OracleError:
            want = None
        in_place = rng.random() < 0.3
        R = empty(n + 4, dtype)[shift:shift + n]
        C = R if in_place else empty(n + 4, dtype)[shift:shift + n]
        if n:
            R.copy_(dev_bits(ref, dtype))
            if not in_place:
                C.copy_(R)
        print("perturb fuzz", k, dtype, op, n, shift, in_place, flush=True)
        try:
            sv.perturb(R, C, seed, stream, op, idx=idx, **kw)
            got = bits(C)
        except sv.SVError:
            got = None
        if want is None:
            assert got is None, (k, dtype, op, "the library accepted what the oracle refuses")
            refused += 1
        else:
            assert got is not None, (k, dtype, op, "the library refused what the oracle accepts")
            assert np.array_equal(got, want.view(got.dtype)), (k, dtype, op, n, shift, in_place)
            done += 1
    print("perturb fuzz: %d steps compared, %d refused by both" % (done, refused), flush=True)
    assert done >= 30


EXTREME = [("ulp", dict(p=-0.1)), ("ulp", dict(p=1.5)), ("ulp", dict(p=float("nan"))), ("ulp", dict(p=1.0)),
           ("scale", dict(p=1.0, value=float("inf"))), ("scale", dict(p=1.0, value=float("nan"))),
           ("scale", dict(p=1.0, value=-1e-3)), ("scale", dict(p=1.0, value=0.0)), ("scale", dict(p=1.0, value=3e38)),
           ("add_at", dict(value=float("inf"))), ("add_at", dict(value=float("nan"))), ("add_at", dict(value=1e300)),
           ("special_flip", dict(p=1.0)), ("set_at", dict(bits=0xFFFFFFFF))]


@pytest.mark.parametrize("dtype", TYPES)
@pytest.mark.parametrize("op,kw", EXTREME)
def test_extreme_plans_agree_with_the_oracle(oracle, dtype, op, kw):
    """Probabilities outside [0, 1] or NaN, infinite and NaN widths and deltas:
    refused by the library exactly where the oracle refuses them, otherwise
    the oracle's bits."""
    n = 5000
    ref = _reference(oracle, np.random.default_rng(9500), dtype, n)
    idx = np.array([0, 17, 4999], dtype=np.uint64) if op in ("add_at", "set_at", "fault_at") else None
    try:
        want = oracle.perturb(8, 9, dtype, op, ref, ref.copy(), idx=idx, **kw)
    except oracle.OracleError:
        want = None
    R = dev_bits(ref, dtype)
    C = R.clone()
    try:
        sv.perturb(R, C, 8, 9, op, idx=idx, **kw)
        got = bits(C)
    except sv.SVError:
        got = None
    if want is None:
        assert got is None, "the library accepted what the oracle refuses"
    else:
        assert got is not None, "the library refused what the oracle accepts"
        assert np.array_equal(got, want.view(got.dtype))

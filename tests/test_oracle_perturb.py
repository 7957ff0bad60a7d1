"""Pins of the oracle's candidate derivation (test-workload support).

The candidates stand in for kernel outputs K(x) that are correct up to
rounding, or carry known faults, so that Eq. (1) has something to find.  Each
step is pinned against numpy / torch library routines, a brute-force order of
all bf16 values, and the Philox words that select elements.
"""
import math

import numpy as np
import pytest
import torch

F32_EDGE = np.array([0, 0x80000000, 1, 0x80000001, 0x007FFFFF, 0x807FFFFF, 0x00800000, 0x3F800000,
                     0xBF800000, 0x7F7FFFFF, 0xFF7FFFFF, 0x7F800000, 0xFF800000], dtype=np.uint32)


def f32(bits):
    return np.asarray(bits, dtype=np.uint32).view(np.float32)


def test_next_f32_matches_numpy_nextafter(oracle):
    rng = np.random.default_rng(1)
    bits = np.concatenate([F32_EDGE, rng.integers(0, 2 ** 32, 200000, dtype=np.uint64).astype(np.uint32)])
    bits = bits[(bits & 0x7FFFFFFF) <= 0x7F800000]
    for up in (0, 1):
        want = np.nextafter(f32(bits), np.float32(np.inf if up else -np.inf)).view(np.uint32)
        got = np.array([oracle.next_f32(int(b), up) for b in bits], dtype=np.uint32)
        assert np.array_equal(got, want)
    for nan in (0x7FC00000, 0xFFC00001, 0x7F800001):
        assert oracle.next_f32(nan, 1) == nan and oracle.next_f32(nan, 0) == nan


def test_next_bf16_by_brute_force_order(oracle):
    pats = np.arange(1 << 16, dtype=np.uint32)
    vals = f32(pats << 16).astype(np.float64)
    ok = ~np.isnan(vals)
    order = np.unique(vals[ok])                       # all distinct bf16 values, sorted
    for p in pats[ok]:
        x = vals[p]
        for up in (0, 1):
            got = oracle.next_bf16(int(p), up)
            g = float(f32(np.uint32(got) << 16))
            k = np.searchsorted(order, x)
            if up:
                want = x if x == np.inf else order[k + 1]
            else:
                want = x if x == -np.inf else order[k - 1]
            assert g == want, (hex(p), up)
            if g == 0:   # a step onto zero keeps the sign of the start
                assert (got >> 15) == (p >> 15)


def test_ulp_step_selection_and_direction(oracle):
    n = 1 << 16
    ref = oracle.synth(0, 0, "f32", "normal", oracle.dist_params(mean=0.0, std=1.0), n)
    stream = (1 << 63) | (1 << 32)
    p = 0.05
    cand = oracle.perturb(0, stream, "f32", "ulp", ref, p=p)
    w = oracle.philox_blocks(0, stream, 0, n)
    sel = w[:, 0].astype(np.uint64) < math.floor(p * 2 ** 32)
    up = (w[:, 1] >> 31) == 1
    assert np.array_equal(cand[~sel], ref[~sel])
    want = np.where(up, np.nextafter(f32(ref), np.float32(np.inf)),
                    np.nextafter(f32(ref), np.float32(-np.inf))).view(np.uint32)
    assert np.array_equal(cand[sel], want[sel])
    assert abs(sel.sum() - n * p) < 5 * math.sqrt(n * p * (1 - p))


def test_scale_step_exact(oracle):
    n = 1 << 14
    ref = oracle.synth(0, 3, "bf16", "uniform", oracle.dist_params(a=-4.0, b=4.0), n)
    stream = (1 << 63) | (2 << 32) | 3
    cand = oracle.perturb(0, stream, "bf16", "scale", ref, p=1.0, value=2.0 ** -9)
    w = oracle.philox_blocks(0, stream, 0, n)
    # u = (w2 >> 8) 2^-32 - 2^-9 is exact in fp32; 1 + u, b * s in fp32 (numpy), then bf16 (torch)
    u = ((w[:, 2] >> 8).astype(np.float64) * 2.0 ** -32 - 2.0 ** -9).astype(np.float32)
    assert np.array_equal(u.astype(np.float64), (w[:, 2] >> 8).astype(np.float64) * 2.0 ** -32 - 2.0 ** -9)
    s = np.float32(1) + u
    b = f32(ref.astype(np.uint32) << 16)
    x = b * s
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(cand, want)
    c = f32(cand.astype(np.uint32) << 16).astype(np.float64)
    bb = b.astype(np.float64)
    assert np.all(np.abs(c - bb) <= np.abs(bb) * (2.0 ** -9 + 2.0 ** -8) + 1e-30)


def test_special_flip(oracle):
    n = 1 << 16
    sp = dict(mean=0.0, std=1e3, p_nan=0.1, p_inf=0.05, p_denorm=0.1, p_zero=0.1)
    ref = oracle.synth(0, 0, "f32", "special", oracle.dist_params(**sp), n)
    stream = (1 << 63) | (3 << 32)
    cand = oracle.perturb(0, stream, "f32", "special_flip", ref, p=0.5)
    w = oracle.philox_blocks(0, stream, 0, n)
    sel = w[:, 0].astype(np.uint64) < 2 ** 31
    zero = (ref & 0x7FFFFFFF) == 0
    nan = (ref & 0x7FFFFFFF) > 0x7F800000
    assert np.array_equal(cand[sel & zero], ref[sel & zero] ^ np.uint32(0x80000000))
    m = w[:, 1] & 0x3FFFFF
    m = np.where(m == 0, 1, m).astype(np.uint32)
    assert np.array_equal(cand[sel & nan], ref[sel & nan] ^ m[sel & nan])
    assert np.all(np.isnan(f32(cand[nan]))) and np.all(cand[nan] & 0x400000)
    assert np.all(cand[sel & nan] != ref[sel & nan])
    keep = ~(sel & (zero | nan))
    assert np.array_equal(cand[keep], ref[keep])
    assert 0.4 < (sel & zero).sum() / zero.sum() < 0.6


def test_index_steps(oracle):
    ref = oracle.synth(0, 0, "f32", "uniform", oracle.dist_params(a=-1.0, b=1.0), 1000)
    idx = np.array([3, 999, 0, 500], dtype=np.uint64)
    c = oracle.perturb(0, 0, "f32", "add_at", ref, value=1e-3, idx=idx)
    r = f32(ref)
    want = r.copy()
    want[idx.astype(np.int64)] = r[idx.astype(np.int64)] + np.float32(1e-3)
    assert np.array_equal(f32(c), want)
    c = oracle.perturb(0, 0, "f32", "set_at", ref, bits=0x7FC00000, idx=idx)
    assert np.all(c[idx.astype(np.int64)] == 0x7FC00000)
    assert np.sum(c != ref) == 4
    c = oracle.perturb(0, 0, "f32", "fault_at", ref, idx=idx)
    x = r[idx.astype(np.int64)]
    assert np.array_equal(f32(c)[idx.astype(np.int64)], x + (np.float32(1) + np.abs(x)))
    iref = np.array([5, -7, 2 ** 31 - 1, -2 ** 31], dtype=np.int32).view(np.uint32)
    c = oracle.perturb(0, 0, "i32", "fault_at", iref, idx=np.arange(4, dtype=np.uint64))
    assert list(c.view(np.int32)) == [6, -6, -2 ** 31, -2 ** 31 + 1]


def test_window_equals_slice_of_full(oracle):
    n = 4096
    ref = oracle.synth(0, 0, "f32", "special",
                       oracle.dist_params(mean=0.0, std=1.0, p_nan=0.2, p_inf=0.1, p_denorm=0.1,
                                          p_zero=0.2), n)
    idx = np.array([10, 1000, 4000], dtype=np.uint64)
    for op, kw in [("ulp", dict(p=0.3)), ("special_flip", dict(p=0.5)),
                   ("set_at", dict(bits=0x7F800000, idx=idx)), ("fault_at", dict(idx=idx))]:
        full = oracle.perturb(1, 2, "f32", op, ref, **kw)
        for off, m in [(0, 7), (999, 5), (3999, 97)]:
            part = oracle.perturb(1, 2, "f32", op, ref[off:off + m], offset=off, **kw)
            assert np.array_equal(part, full[off:off + m]), (op, off)


def test_fault_step_on_nan_and_infinite_references(oracle):
    """The fault step x + (1 + |x|) on references that are not finite, per
    element format: +Inf stays +Inf; -Inf gives the invalid operation's quiet
    NaN with the sign bit set and no payload; a NaN gives its magnitude with
    the quiet bit set (signalling NaNs quieted, sign cleared, payload kept),
    then the format's NaN rule for bf16 and fp16 (their fp32 value narrowed).
    Finite references: the sum in the element's arithmetic (numpy)."""
    cases = {
        "f64": (np.uint64, np.float64, 0x7FF0000000000000, 0xFFF0000000000000, 0xFFF8000000000000, 1 << 51,
                [0x7FF8000000000000, 0xFFF8000000000000, 0x7FF8000000000001, 0xFFF4000000000000,
                 0x7FF0000000000001, 0xFFF0000000000123]),
        "f32": (np.uint32, np.float32, 0x7F800000, 0xFF800000, 0xFFC00000, 1 << 22,
                [0x7FC00000, 0xFFC00000, 0x7FC00001, 0xFFA00000, 0x7F800001, 0xFF800123]),
    }
    for dtype, (st, ft, pinf, ninf, inv, quiet, nans) in cases.items():
        finite = np.array([0.0, -0.0, 1.0, -1.5, 3e-300 if dtype == "f64" else 3e-38, -7.25], dtype=ft)
        ref = np.concatenate([np.array([pinf, ninf] + nans, dtype=st), finite.view(st)])
        c = oracle.perturb(0, 0, dtype, "fault_at", ref, idx=np.arange(ref.size, dtype=np.uint64))
        sign = st(1) << st(8 * np.dtype(st).itemsize - 1)
        assert c[0] == pinf and c[1] == inv
        for k, v in enumerate(nans):
            assert c[2 + k] == (st(v) & ~sign) | st(quiet), (dtype, hex(v), hex(int(c[2 + k])))
        x = finite
        assert np.array_equal(c[2 + len(nans):].view(ft), x + (ft(1) + np.abs(x)))
    # bf16 and fp16: the fp32 result narrowed by the format's rules
    for dtype, nan_in, want in (("bf16", [0xFF80, 0xFFC0, 0xFFA0, 0x7F81], [0xFFC0, 0x7FC0, 0x7FE0, 0x7FC1]),
                                ("f16", [0xFC00, 0xFE00, 0xFD00, 0x7C01], [0xFE00, 0x7E00, 0x7F00, 0x7E01])):
        ref = np.array(nan_in, dtype=np.uint16)
        c = oracle.perturb(0, 0, dtype, "fault_at", ref, idx=np.arange(ref.size, dtype=np.uint64))
        assert [int(v) for v in c] == want, (dtype, [hex(int(v)) for v in c])


def test_scale_and_add_need_a_finite_fp32_value(oracle):
    """The scale width and the added delta enter as fp32 values (fp32(1 + u)
    with |u| <= value, fp32(y) + fp32(value)); a value that is NaN, infinite,
    or overflows fp32 is refused, and the largest finite fp32 is accepted."""
    ref = np.array([0x3F800000, 0x40000000], np.uint32)
    idx = np.array([1], np.uint64)
    for op in ("scale", "add_at"):
        for bad in (float("nan"), float("inf"), -float("inf"), 1e300, -3.5e38):
            with pytest.raises(oracle.OracleError):
                oracle.perturb(0, 0, "f32", op, ref, p=1.0, value=bad, idx=idx)
        oracle.perturb(0, 0, "f32", op, ref, p=1.0, value=float(np.finfo(np.float32).max), idx=idx)

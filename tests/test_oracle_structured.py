"""Pins of the oracle's permutation distribution (structured inputs): element i
of a tensor is lo + pi(i), pi a seeded bijection of [0, N), N = hi - lo + 1
(a ten-round Feistel network and a rotation, with cycle walking, keys from
the tensor's Philox sequence).  What fixes it without another implementation: it is a
bijection for every N (brute force), windows are slices, shorter tensors are
samples without replacement, it is invertible by the rounds run backwards
where no walk happens, and the orders it produces are uniform."""
import itertools
import math

import numpy as np
import pytest


def _perm(oracle, seed, stream, lo, hi, n, dtype="i64", offset=0):
    v = oracle.synth(seed, stream, dtype, "permutation", oracle.dist_params(lo=lo, hi=hi), n, offset=offset)
    return v.view(np.int64) if dtype == "i64" else v.astype(np.int64) if dtype == "u8" else v.view(np.int32).astype(np.int64)


@pytest.mark.parametrize("N", [1, 2, 3, 4, 5, 7, 8, 9, 16, 17, 255, 256, 1000, 4096, 65537, 100003])
def test_is_a_bijection_of_the_domain(oracle, N):
    for lo, dtype in ((0, "i64"), (-37, "i32"), (5, "i64")):
        v = _perm(oracle, 3, 9, lo, lo + N - 1, N, dtype)
        assert np.array_equal(np.sort(v), np.arange(lo, lo + N)), (N, lo)
    if N <= 256:
        assert np.array_equal(np.sort(_perm(oracle, 3, 9, 0, N - 1, N, "u8")), np.arange(N))


def test_windows_are_slices_and_short_tensors_sample_without_replacement(oracle):
    N = 50_000
    full = _perm(oracle, 11, 2, 100, 100 + N - 1, N)
    for off, m in ((0, 1), (1, 17), (12_345, 1000), (N - 7, 7)):
        assert np.array_equal(_perm(oracle, 11, 2, 100, 100 + N - 1, m, offset=off), full[off:off + m])
    idx = np.array([0, 5, N - 1, 777], np.uint64)
    at = oracle.synth_at(11, 2, "i64", "permutation", oracle.dist_params(lo=100, hi=100 + N - 1), idx).view(np.int64)
    assert np.array_equal(at, full[idx.astype(np.int64)])
    sample = _perm(oracle, 4, 4, -2 ** 40, 2 ** 40, 20_000)             # 20,000 of 2^41 + 1 values
    assert np.unique(sample).size == 20_000 and sample.min() >= -2 ** 40 and sample.max() <= 2 ** 40
    with pytest.raises(RuntimeError):
        _perm(oracle, 11, 2, 100, 100 + N - 1, 8, offset=N - 7)         # past the N values
    with pytest.raises(RuntimeError):
        _perm(oracle, 0, 0, 0, 2 ** 61, 4)                              # N above 2^60
    with pytest.raises(RuntimeError):
        _perm(oracle, 0, 0, 0, 256, 4, "u8")
    with pytest.raises(RuntimeError):
        oracle.synth(0, 0, "f32", "permutation", oracle.dist_params(lo=0, hi=9), 4)


def _lowbias32(x):
    x ^= x >> 16
    x = (x * 0x7FEB352D) & 0xFFFFFFFF
    x ^= x >> 15
    x = (x * 0x846CA68B) & 0xFFFFFFFF
    x ^= x >> 16
    return x


def test_inverted_by_the_rounds_run_backwards(oracle):
    # N = 2^(2h): no walk, so pi is the word permutation itself: subtract the
    # rotation K_10, then undo round r (from the last), which maps
    # (L', R') = (R, L ^ f(R)) back to (L, R)
    for h, seed in ((1, 5), (3, 6), (8, 7), (11, 8)):
        N = 1 << (2 * h)
        n = min(N, 5000)
        v = _perm(oracle, seed, 1, 0, N - 1, n)
        key = oracle.philox_blocks(seed, 1, 0, 3).reshape(-1).astype(np.uint64)[:11]
        mask = (1 << h) - 1
        for i, x in enumerate(v.tolist()):
            x = (x - int(key[10])) % N
            l, r = x >> h, x & mask
            for k in reversed(range(10)):
                l, r = r ^ (_lowbias32((l ^ int(key[k])) & 0xFFFFFFFF) & mask), l
            assert (l << h) | r == i, (h, i)


def test_orders_are_uniform(oracle):
    # all 120 orders of 5 values over 12,000 streams: chi-square with 119 degrees
    # of freedom (mean 119, sd 15.4); six Feistel rounds alone (even
    # permutations of the words) gave 516 here, six and the rotation 167
    counts = {p: 0 for p in itertools.permutations(range(5))}
    for s in range(12_000):
        counts[tuple(_perm(oracle, 21, s, 0, 4, 5).tolist())] += 1
    chi2 = sum((c - 100) ** 2 / 100 for c in counts.values())
    assert chi2 < 119 + 4 * 15.4, chi2
    # a large domain: positions and values uncorrelated, few fixed points (Poisson(1) on average)
    N = 1 << 20
    v = _perm(oracle, 5, 5, 0, N - 1, N)
    assert abs(np.corrcoef(np.arange(N), v)[0, 1]) < 0.01
    assert int((v == np.arange(N)).sum()) <= 8
    assert not np.array_equal(v, _perm(oracle, 5, 6, 0, N - 1, N))     # another stream, another order

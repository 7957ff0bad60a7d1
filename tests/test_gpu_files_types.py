"""Test-data files of every element type across the 64 MiB chunk boundary.

For each of the seven types: sv_synth_file writes a tensor a few elements
longer than one 64 MiB chunk (a random tail length), whose bytes must be the
oracle's synthesis; then sv_compare_file checks it against a candidate file
that differs in a few seeded places, one of them in the second chunk, and the
report must be the oracle's.
"""
import numpy as np
import pytest

import paper_2609_00058_amd as sv

pytestmark = pytest.mark.gpu

CHUNK = 64 << 20
ITEM = {"f32": 4, "bf16": 2, "i32": 4, "f16": 2, "f64": 8, "u8": 1, "i64": 8}
STORAGE = {"f32": np.uint32, "bf16": np.uint16, "i32": np.uint32, "f16": np.uint16, "f64": np.uint64,
           "u8": np.uint8, "i64": np.uint64}
SPECIAL = dict(mean=0.0, std=1e3, p_nan=0.01, p_inf=0.01, p_denorm=0.01, p_zero=0.01)


@pytest.mark.parametrize("dtype", list(ITEM))
def test_file_round_trip_across_the_chunk_boundary(oracle, tmp_path, dtype):
    rng = np.random.default_rng(9400 + ITEM[dtype] + len(dtype))
    n = CHUNK // ITEM[dtype] + int(rng.integers(1, 40))
    if dtype in ("i32", "u8", "i64"):
        dist, params = "int_range", dict(lo=0, hi=200) if dtype == "u8" else dict(lo=-10 ** 6, hi=10 ** 6)
    else:
        dist, params = "special", SPECIAL
    ref_path, cand_path = tmp_path / "ref.bin", tmp_path / "cand.bin"
    print("file", dtype, n, flush=True)
    sv.synth_file(str(ref_path), n, 5, 6, dtype, dist, **params)
    want = oracle.synth(5, 6, dtype, dist, oracle.dist_params(**params), n)
    got = np.fromfile(ref_path, dtype=STORAGE[dtype])
    assert got.size == n and np.array_equal(got, want)
    cand = want.copy()
    where = np.unique(np.concatenate([rng.integers(0, n, 5), [n - 1, CHUNK // ITEM[dtype] + 1]]))
    cand[where] ^= STORAGE[dtype](1)                  # the lowest bit of the value or integer
    cand.tofile(cand_path)
    for rtol, atol, eqn in ((0.0, 0.0, False), (1e-3, 1e-6, True)):
        rep = sv.compare_file(str(ref_path), str(cand_path), n, dtype, rtol, atol, eqn)
        w = oracle.compare(want, cand, dtype, rtol, atol, eqn)
        for k in w:
            if k == "err_sum" and w[k] not in (0.0, float("inf")):
                assert abs(rep[k] - w[k]) <= 1e-12 * abs(w[k]), (dtype, k, rep[k], w[k])
            else:
                assert rep[k] == w[k], (dtype, k, rep[k], w[k])

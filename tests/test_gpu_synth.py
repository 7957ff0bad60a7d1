"""GPU parity of sv_synth and sv_perturb against the CPU oracle (bit-exact).

Sizes span several workgroup tiles and ragged tails; outputs that are not
16-byte aligned exercise the one-element-per-thread path; full-size tensors
are checked on sampled elements the oracle computes one by one.
"""
import numpy as np
import pytest
import torch

import paper_2609_00058_amd as sv
from gpu_run import bits, bits_at, empty

pytestmark = pytest.mark.gpu

SPECIAL = dict(mean=0.0, std=1e3, p_nan=0.01, p_inf=0.005, p_denorm=0.01, p_zero=0.01)
SPECIAL_HEAVY = dict(mean=5.0, std=10.0, p_nan=0.2, p_inf=0.1, p_denorm=0.2, p_zero=0.2)
# about 60 % of the 16-byte vectors hold a candidate: a wave's list of them fills up part way through a group
SPECIAL_MID = dict(mean=1.0, std=3.0, p_nan=0.05, p_inf=0.05, p_denorm=0.05, p_zero=0.05)
# every element special: the last class threshold is 2^32 (no class word keeps its normal value)
SPECIAL_ALL = dict(mean=0.0, std=1.0, p_nan=0.25, p_inf=0.25, p_denorm=0.25, p_zero=0.25)
CASES = [
    ("uniform", "f32", dict(a=-1.0, b=1.0)),
    ("uniform", "f32", dict(a=-3.0, b=7.5)),
    ("uniform", "bf16", dict(a=-4.0, b=4.0)),
    ("uniform", "bf16", dict(a=-3.0, b=7.5)),
    ("normal", "f32", dict(mean=0.0, std=1.0)),
    ("normal", "f32", dict(mean=5.0, std=10.0)),
    ("normal", "bf16", dict(mean=5.0, std=10.0)),
    ("int_range", "i32", dict(lo=-(1 << 20), hi=1 << 20)),
    ("int_range", "i32", dict(lo=-2 ** 31, hi=2 ** 31 - 1)),
    ("int_range", "i32", dict(lo=7, hi=7)),
    ("special", "f32", SPECIAL),
    ("special", "f32", SPECIAL_HEAVY),
    ("special", "bf16", SPECIAL_HEAVY),
    ("special", "f32", SPECIAL_MID),
    ("special", "f32", SPECIAL_ALL),
    ("special", "f32", dict(mean=0.0, std=1.0, p_nan=1.0)),
    # the 16-bit types through the listing kernel: two blocks per 16-byte vector
    ("special", "bf16", SPECIAL),
    ("special", "bf16", SPECIAL_MID),
    ("special", "bf16", SPECIAL_ALL),
    ("special", "bf16", dict(mean=0.0, std=1.0, p_nan=1.0)),
    ("special", "bf16", dict(mean=0.0, std=1e38)),
    ("special", "f16", SPECIAL_HEAVY),
    ("special", "f16", SPECIAL_MID),
    ("special", "f16", SPECIAL_ALL),
    ("special", "f16", dict(mean=0.0, std=1.0, p_inf=1.0)),
    ("special", "f16", dict(mean=0.0, std=1e5, p_denorm=0.02)),
    # fp16 uniform and normal values: two blocks per 16-byte vector, hardware conversions
    ("uniform", "f16", dict(a=-4.0, b=4.0)),
    ("uniform", "f16", dict(a=60000.0, b=65504.0)),
    ("normal", "f16", dict(mean=5.0, std=10.0)),
    ("normal", "f16", dict(mean=0.0, std=3e4)),
    # uint8: four blocks per 16-byte vector, one 32-bit word per element
    ("int_range", "u8", dict(lo=0, hi=255)),
    ("int_range", "u8", dict(lo=3, hi=202)),
    ("int_range", "u8", dict(lo=7, hi=7)),
    # fp64: one block per two 16-byte vectors, every value widened with the NaN rule
    ("special", "f64", SPECIAL),
    ("special", "f64", SPECIAL_MID),
    ("special", "f64", SPECIAL_ALL),
    ("special", "f64", dict(mean=0.0, std=1.0, p_nan=1.0)),
    ("special", "f64", dict(mean=-3e38, std=1e38, p_inf=0.1)),
]
SIZES = [1, 3, 4, 5, 8, 17, 1000, 4099, 65543, (1 << 20) + 3]


def _diff(got, want):
    bad = np.nonzero(got != want)[0]
    return "first diff at %d of %d: got %#x want %#x" % (bad[0], bad.size, got[bad[0]], want[bad[0]]) \
        if bad.size else ""


@pytest.mark.parametrize("dist,dtype,params", CASES)
def test_synth_bit_exact(oracle, dist, dtype, params):
    for n in SIZES:
        seed, stream = 0xDEADBEEF12345678, (1 << 63) | n
        print("synth", dist, dtype, n, flush=True)
        g = empty(n, dtype)
        sv.synth(g, seed, stream, dist, **params)
        want = oracle.synth(seed, stream, dtype, dist, oracle.dist_params(**params), n)
        got = bits(g)
        assert np.array_equal(got, want), _diff(got, want)


@pytest.mark.parametrize("dist,dtype,params", [CASES[0], CASES[2], CASES[3], CASES[5], CASES[7], CASES[11], CASES[12]])
def test_synth_unaligned_outputs_and_guard(oracle, dist, dtype, params):
    n = 5003
    per = 8 if dtype == "bf16" else 4
    for off in range(1, per):
        big = empty(n + 2 * per, dtype)
        big.view(torch.int16 if dtype == "bf16" else torch.int32).fill_(0x5A5A)
        view = big[off:off + n]
        print("synth unaligned", dist, dtype, off, flush=True)
        sv.synth(view, 9, 4, dist, **params)
        want = oracle.synth(9, 4, dtype, dist, oracle.dist_params(**params), n)
        allb = bits(big)
        assert np.array_equal(allb[off:off + n], want), _diff(allb[off:off + n], want)
        assert np.all(allb[:off] == 0x5A5A) and np.all(allb[off + n:] == 0x5A5A)


@pytest.mark.parametrize("dist,dtype,params", [("normal", "f32", dict(mean=5.0, std=10.0)),
                                               ("special", "f32", SPECIAL), ("special", "f32", SPECIAL_MID),
                                               ("special", "bf16", SPECIAL), ("special", "bf16", SPECIAL_MID),
                                               ("special", "f16", SPECIAL), ("special", "f16", SPECIAL_ALL),
                                               ("special", "f64", SPECIAL), ("special", "f64", SPECIAL_MID),
                                               ("uniform", "f16", dict(a=-1.0, b=3.0)),
                                               ("normal", "f16", dict(mean=1.0, std=2.0)),
                                               ("int_range", "u8", dict(lo=10, hi=250))])
def test_synth_far_window_with_64_bit_block_indices(oracle, dist, dtype, params):
    # a window past element 2^40: Philox block indices above 2^32, so the kernels index in 64 bits;
    # large enough for whole tiles and a ragged last one
    n, off = (1 << 20) + 3, (1 << 40) + 12
    print("far window", dist, dtype, params, flush=True)
    g = empty(n, dtype)
    sv.synth_window(g, 11, 5, dist, off, **params)
    want = oracle.synth(11, 5, dtype, dist, oracle.dist_params(**params), n, off)
    got = bits(g)
    assert np.array_equal(got, want), _diff(got, want)


@pytest.mark.parametrize("dist,dtype,params", [("normal", "f32", dict(mean=0.0, std=1.0)), ("uniform", "bf16", dict(a=-4.0, b=4.0)),
                                               ("special", "f32", SPECIAL_MID), ("special", "bf16", SPECIAL),
                                               ("special", "f16", SPECIAL_MID), ("special", "f64", SPECIAL),
                                               ("uniform", "f16", dict(a=-4.0, b=4.0)),
                                               ("normal", "f16", dict(mean=0.0, std=1.0)),
                                               ("int_range", "u8", dict(lo=0, hi=99))])
def test_synth_window_across_block_2_to_the_32(oracle, dist, dtype, params):
    # a window whose Philox block indices cross 2^32 (element 2^34) part way through: the kernels must
    # take 64-bit indices for the whole launch; ragged at both ends of a tile
    n, off = (1 << 20) + 3, (1 << 34) - (1 << 19) + 4
    print("window across block 2^32", dist, dtype, flush=True)
    g = empty(n, dtype)
    sv.synth_window(g, 21, 22, dist, off, **params)
    want = oracle.synth(21, 22, dtype, dist, oracle.dist_params(**params), n, off)
    got = bits(g)
    assert np.array_equal(got, want), _diff(got, want)


def test_synth_is_deterministic_and_empty_ok():
    a, b = empty(1 << 20, "f32"), empty(1 << 20, "f32")
    sv.synth(a, 1, 2, "normal", mean=0.0, std=1.0)
    sv.synth(b, 1, 2, "normal", mean=0.0, std=1.0)
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    sv.synth(empty(0, "f32"), 1, 2, "normal", mean=0.0, std=1.0)


def test_synth_rejects_bad_arguments():
    g = empty(16, "f32")
    with pytest.raises(sv.SVError) as e:
        sv.synth(g, 0, 0, "int_range", lo=0, hi=5)
    assert e.value.code == sv.SV_ERR_UNSUPPORTED
    with pytest.raises(sv.SVError) as e:
        sv.synth(g, 0, 0, "uniform", a=1.0, b=1.0)
    assert e.value.code == sv.SV_ERR_INVALID_ARG
    with pytest.raises(sv.SVError):
        sv.synth(g, 0, 0, "special", p_nan=0.7, p_inf=0.7)


@pytest.mark.parametrize("dist,dtype,n,params", [
    ("normal", "f32", 1 << 26, dict(mean=0.0, std=1.0)),
    ("special", "f32", 1 << 30, SPECIAL),
    ("uniform", "bf16", 1 << 24, dict(a=-4.0, b=4.0)),
])
def test_synth_full_size_sampled(oracle, dist, dtype, n, params):
    print("synth full", dist, dtype, n, flush=True)
    g = empty(n, dtype)
    sv.synth(g, 0, 0, dist, **params)
    rng = np.random.default_rng(n)
    idx = np.unique(np.concatenate([np.arange(4096), np.arange(n - 4096, n),
                                    rng.integers(0, n, 60000)])).astype(np.uint64)
    got = bits_at(g, idx)
    want = oracle.synth_at(0, 0, dtype, dist, oracle.dist_params(**params), idx)
    assert np.array_equal(got, want), _diff(got, want)
    del g
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dist,dtype,params", [("normal", "f32", dict(mean=0.0, std=1.0)),
                                               ("special", "f32", SPECIAL), ("special", "bf16", SPECIAL),
                                               ("special", "f16", SPECIAL_MID), ("special", "f64", SPECIAL),
                                               ("normal", "f16", dict(mean=0.0, std=1.0))])
def test_synth_far_window_of_1_gib_sampled(oracle, dist, dtype, params):
    # 1 GiB of values (2^28 + 5 fp32, 2^29 + 5 bf16 / fp16, 2^27 + 5 fp64) past element 2^40: 64-bit
    # block indices and the non-temporal stores of outputs of 1 GiB or more, together; sampled against
    # the oracle element by element
    n, off = (1 << 30) // {"f32": 4, "bf16": 2, "f16": 2, "f64": 8}[dtype] + 5, (1 << 40) + 12
    print("far window 1 GiB", dist, dtype, flush=True)
    g = empty(n, dtype)
    sv.synth_window(g, 3, 9, dist, off, **params)
    rng = np.random.default_rng(77)
    idx = np.unique(np.concatenate([np.arange(4096), np.arange(n - 4096, n),
                                    rng.integers(0, n, 60000)])).astype(np.uint64)
    got = bits_at(g, idx)
    want = oracle.synth_at(3, 9, dtype, dist, oracle.dist_params(**params), idx + np.uint64(off))
    assert np.array_equal(got, want), _diff(got, want)
    del g
    torch.cuda.empty_cache()


def test_synth_batched_matches_single_calls_and_oracle(oracle):
    rng = np.random.default_rng(12)
    jobs, singles = [], []
    keep = []
    for k, (dist, dtype, params) in enumerate(CASES * 3):
        n = int(rng.choice([0, 1, 3, 8, 255, 256 * 4 + 1, 70001, 1 << 20]))
        off = int(rng.integers(0, 3)) if k % 4 == 0 else 0          # some outputs not 16-byte aligned
        big = empty(n + 8, dtype)
        out = big[off:off + n]
        ref = empty(n, dtype)
        keep += [big, ref]
        jobs.append((out, 5 + k, (1 << 63) | k, dist, params))
        singles.append((ref, 5 + k, (1 << 63) | k, dist, params))
    print("synth batched", len(jobs), flush=True)
    sv.synth_batched(jobs)
    for ref, seed, stream, dist, params in singles:
        sv.synth(ref, seed, stream, dist, **params)
    for (out, seed, stream, dist, params), (ref, *_rest) in zip(jobs, singles):
        assert np.array_equal(bits(out), bits(ref))
    for out, seed, stream, dist, params in jobs[:12] + jobs[-12:]:
        dtype = {torch.float32: "f32", torch.bfloat16: "bf16", torch.int32: "i32", torch.float16: "f16",
                 torch.float64: "f64", torch.uint8: "u8"}[out.dtype]
        want = oracle.synth(seed, stream, dtype, dist, oracle.dist_params(**params), out.numel())
        assert np.array_equal(bits(out), want)
    # back-to-back batches reuse the job table: the second must not see the first's jobs
    a, b = empty(5000, "f32"), empty(7000, "bf16")
    sv.synth_batched([(a, 1, 1, "normal", dict(mean=0.0, std=1.0))])
    sv.synth_batched([(b, 2, 2, "uniform", dict(a=-1.0, b=1.0))])
    assert np.array_equal(bits(a), oracle.synth(1, 1, "f32", "normal", oracle.dist_params(mean=0.0, std=1.0), 5000))
    assert np.array_equal(bits(b), oracle.synth(2, 2, "bf16", "uniform", oracle.dist_params(a=-1.0, b=1.0), 7000))


PERTURB = [
    ("f32", "uniform", dict(a=-1.0, b=1.0), "copy", {}),
    ("f32", "normal", dict(mean=0.0, std=1.0), "ulp", dict(p=0.3)),
    ("bf16", "normal", dict(mean=5.0, std=10.0), "ulp", dict(p=0.3)),
    ("f32", "special", SPECIAL_HEAVY, "ulp", dict(p=0.5)),
    ("bf16", "uniform", dict(a=-4.0, b=4.0), "scale", dict(p=1.0, value=2.0 ** -9)),
    ("f32", "normal", dict(mean=5.0, std=10.0), "scale", dict(p=0.7, value=0.25)),
    ("f32", "special", SPECIAL_HEAVY, "special_flip", dict(p=0.5)),
    ("bf16", "special", SPECIAL_HEAVY, "special_flip", dict(p=0.5)),
    ("i32", "int_range", dict(lo=-100, hi=100), "copy", {}),
]


@pytest.mark.parametrize("dtype,dist,params,op,kw", PERTURB)
def test_perturb_elementwise_bit_exact(oracle, dtype, dist, params, op, kw):
    for n in (1, 7, 4099, (1 << 20) + 3):
        print("perturb", op, dtype, n, flush=True)
        ref = empty(n, dtype)
        sv.synth(ref, 3, 1, dist, **params)
        cand = empty(n, dtype)
        stream = (1 << 63) | (5 << 32) | n
        sv.perturb(ref, cand, 11, stream, op, **kw)
        r = oracle.synth(3, 1, dtype, dist, oracle.dist_params(**params), n)
        want = oracle.perturb(11, stream, dtype, op, r, np.empty_like(r), **kw)
        got = bits(cand)
        assert np.array_equal(got, want), _diff(got, want)


@pytest.mark.parametrize("dtype,dist,params", [("f32", "normal", dict(mean=5.0, std=10.0)),
                                               ("bf16", "uniform", dict(a=-4.0, b=4.0)),
                                               ("i32", "int_range", dict(lo=-(1 << 20), hi=1 << 20))])
def test_perturb_index_ops_bit_exact(oracle, dtype, dist, params):
    n = 100003
    rng = np.random.default_rng(4)
    idx = np.concatenate([[0, n - 1], rng.choice(n, 300, replace=False)]).astype(np.uint64)
    ref = empty(n, dtype)
    sv.synth(ref, 0, 7, dist, **params)
    r = oracle.synth(0, 7, dtype, dist, oracle.dist_params(**params), n)
    ops = [("set_at", dict(bits=0x7FC00000)), ("fault_at", {})]
    if dtype != "i32":
        ops.append(("add_at", dict(value=1e-3)))
    for op, kw in ops:
        print("perturb index", op, dtype, flush=True)
        cand = ref.clone()
        sv.perturb(ref, cand, 0, 0, op, idx=idx, **kw)
        want = oracle.perturb(0, 0, dtype, op, r, r.copy(), idx=idx, **kw)
        got = bits(cand)
        assert np.array_equal(got, want), _diff(got, want)
    with pytest.raises(sv.SVError):
        sv.perturb(ref, ref.clone(), 0, 0, "set_at", idx=[n])


def test_normal_transform_building_blocks_exhaustive(oracle):
    # every 24-bit input of ln, the Box-Muller radius, sin and cos: GPU bits == oracle bits
    k = np.arange(1 << 24, dtype=np.uint32)
    kin = torch.from_numpy(k.view(np.int32)).to("cuda")
    out = torch.empty_like(kin)
    want = {
        "ln": oracle.ln_f32_n(((k.astype(np.float64) + 1) * 2.0 ** -24).astype(np.float32)).view(np.uint32),
        "radius": oracle.radius_f32_n(k).view(np.uint32),
    }
    s, c = oracle.sincos_2pi_f32_n(k)
    want["sin"], want["cos"] = s.view(np.uint32), c.view(np.uint32)
    for which in ("ln", "radius", "sin", "cos"):
        print("transform", which, flush=True)
        sv.eval_transform(which, kin, out)
        got = out.cpu().numpy().view(np.uint32)
        assert np.array_equal(got, want[which]), (which, _diff(got, want[which]))

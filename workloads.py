"""Seeded synthetic workloads for the synthesis + check path.

This module is the only thing the GPU path and the CPU oracle share.  It holds
none of the method's arithmetic: no random-number generation of tensor
contents, no distribution transforms, no tolerance checks.  It only states
each workload -- tensor sizes, distributions and their parameters, seeds and
substream ids, tolerances -- and draws the host-side layout of the faults
(which indices, which segments, segment sizes and dtypes) with numpy's PCG64,
seeded per workload.  Both sides then synthesize and derive candidates
themselves from these descriptions.

The six workloads stand in for the paper's benchmark test data (not
available here), following its advice to draw inputs from a broad numeric
range (Sec. 4.2.1; a Gaussian with mean 5 and std 10 is its example, used for
the float segments of the ragged batch).
"""
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

# Substream ids used for candidate derivation: top bit set, a tag in bits
# 32..39, the tensor index below, so they never collide with the tensor
# streams 0, 1, 2, ... used for reference synthesis.
TAG_ULP, TAG_SCALE, TAG_FLIP = 1, 2, 3


def harness_stream(tag: int, index: int) -> int:
    return (1 << 63) | (tag << 32) | index


NAN_F32 = 0x7FC00000
PINF_F32 = 0x7F800000


@dataclass
class TensorSpec:
    n: int
    dtype: str            # "f32" | "bf16" | "i32"
    dist: str             # "uniform" | "normal" | "int_range" | "special"
    params: dict          # keyword arguments of the distribution
    seed: int = 0
    stream: int = 0

    @property
    def itemsize(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    @property
    def nbytes(self) -> int:
        return self.n * self.itemsize


@dataclass
class Step:
    """One candidate-derivation step (applied in order to build the candidate)."""
    op: str               # copy | ulp | scale | special_flip | add_at | set_at | fault_at
    p: float = 0.0
    value: float = 0.0
    bits: int = 0
    idx: Optional[np.ndarray] = None   # uint64 global indices for *_at ops
    seed: int = 0
    stream: int = 0


@dataclass
class Case:
    ref: TensorSpec
    steps: List[Step]
    rtol: float
    atol: float
    equal_nan: bool


@dataclass
class Workload:
    name: str
    cases: List[Case]
    batched: bool
    description: str = ""
    expect: dict = field(default_factory=dict)
    stop_at_first: bool = False     # batched check stops each failing segment at its first mismatch

    def ref_groups(self):
        """The distinct reference tensors (cases may share one: several
        candidates checked against the same output) and, per case, the index
        of its reference among them."""
        uniq, which, seen = [], [], {}
        for c in self.cases:
            key = (c.ref.n, c.ref.dtype, c.ref.dist, tuple(sorted(c.ref.params.items())), c.ref.seed, c.ref.stream)
            if key not in seen:
                seen[key] = len(uniq)
                uniq.append(c.ref)
            which.append(seen[key])
        return uniq, which

    @property
    def total_elems(self) -> int:
        return sum(c.ref.n for c in self.cases)

    @property
    def synth_bytes(self) -> int:
        return sum(r.nbytes for r in self.ref_groups()[0])

    @property
    def compare_bytes(self) -> int:
        return 2 * sum(c.ref.nbytes for c in self.cases)


def _distinct(rng: np.random.Generator, n: int, k: int) -> np.ndarray:
    return rng.choice(n, size=k, replace=False).astype(np.uint64)


def uniform_small(n: int = 65536) -> Workload:
    """65,536 fp32 uniform on [-1, 1) (seed 0, stream 0); the candidate adds
    fp32(1e-3) at 7 distinct seeded indices; rtol 1e-5, atol 1e-8."""
    rng = np.random.Generator(np.random.PCG64(1001))
    idx = _distinct(rng, n, min(7, n))
    ref = TensorSpec(n, "f32", "uniform", dict(a=-1.0, b=1.0))
    steps = [Step("copy"), Step("add_at", value=1e-3, idx=idx)]
    return Workload("uniform_f32_65536", [Case(ref, steps, 1e-5, 1e-8, False)], False,
                    "65,536 fp32 uniform[-1,1); +1e-3 at 7 indices",
                    expect=dict(mismatches=int(idx.size), first=int(idx.min()) if idx.size else -1))


def normal_ulp(n: int = 1 << 26) -> Workload:
    """2^26 fp32 normal(0, 1); candidate = one ulp up or down on a seeded 0.1%
    of elements, then quiet NaN at 16 and +Inf at 16 distinct seeded indices;
    rtol 1e-6, atol 0, equal_nan false."""
    rng = np.random.Generator(np.random.PCG64(1002))
    idx = _distinct(rng, n, min(32, n))
    ref = TensorSpec(n, "f32", "normal", dict(mean=0.0, std=1.0))
    steps = [Step("ulp", p=1e-3, stream=harness_stream(TAG_ULP, 0)),
             Step("set_at", bits=NAN_F32, idx=idx[:16]),
             Step("set_at", bits=PINF_F32, idx=idx[16:32])]
    return Workload("normal_f32_%d" % n, [Case(ref, steps, 1e-6, 0.0, False)], False,
                    "%d fp32 normal(0,1); +-1 ulp on 0.1%%, 16 NaN + 16 +Inf" % n,
                    expect=dict(nan_cand=min(16, idx.size), inf_cand=max(0, idx.size - 16)))


def bf16_batch(count: int = 64, rows: int = 4096, cols: int = 4096) -> Workload:
    """64 bf16 tensors of 4096 x 4096, uniform on [-4, 4) (streams 0..63);
    candidate = bf16(fp32(ref) * (1 + u)), u uniform in [-2^-9, 2^-9);
    rtol = atol = 1e-2; one batched check."""
    cases = []
    for k in range(count):
        ref = TensorSpec(rows * cols, "bf16", "uniform", dict(a=-4.0, b=4.0), stream=k)
        steps = [Step("scale", p=1.0, value=2.0 ** -9, stream=harness_stream(TAG_SCALE, k))]
        cases.append(Case(ref, steps, 1e-2, 1e-2, False))
    return Workload("bf16_batch_%dx%dx%d" % (count, rows, cols), cases, True,
                    "%d bf16 %dx%d uniform[-4,4); x(1+u), |u|<=2^-9" % (count, rows, cols),
                    expect=dict(mismatches=0))


def ragged_batch(count: int = 256, lo_exp: float = 3.0, hi_exp: float = 7.0,
                 fault_frac: float = 0.05) -> Workload:
    """256 ragged fp32 / int32 tensors with sizes floor(10^(3 + 4U)), U
    uniform (log-uniform in [1e3, 1e7]); fp32 ~ normal(5, 10) checked at rtol
    drawn from {1e-3, 1e-5} and atol 1e-6; int32 uniform on [-2^20, 2^20]
    checked exactly; round(5% of count) segments carry one seeded fault."""
    rng = np.random.Generator(np.random.PCG64(1004))
    sizes = np.floor(10.0 ** (lo_exp + (hi_exp - lo_exp) * rng.random(count))).astype(np.int64)
    is_int = rng.random(count) < 0.5
    rtols = np.where(rng.random(count) < 0.5, 1e-3, 1e-5)
    nfault = int(round(fault_frac * count))
    fault_segs = set(int(s) for s in rng.choice(count, size=nfault, replace=False))
    cases, faults = [], {}
    for k in range(count):
        n = int(sizes[k])
        if is_int[k]:
            ref = TensorSpec(n, "i32", "int_range", dict(lo=-(1 << 20), hi=1 << 20), stream=k)
            rtol, atol = 0.0, 0.0
        else:
            ref = TensorSpec(n, "f32", "normal", dict(mean=5.0, std=10.0), stream=k)
            rtol, atol = float(rtols[k]), 1e-6
        steps = [Step("copy")]
        if k in fault_segs and n > 0:
            j = np.array([rng.integers(0, n)], dtype=np.uint64)
            faults[k] = int(j[0])
            steps.append(Step("fault_at", idx=j))
        cases.append(Case(ref, steps, rtol, atol, False))
    return Workload("ragged_batch_%d" % count, cases, True,
                    "%d ragged fp32/int32 tensors, log-uniform sizes, %d faults" % (count, nfault),
                    expect=dict(faults=faults))


def special_stream(n: int = 1 << 30) -> Workload:
    """2^30 fp32 with 1% NaN, 0.5% +-Inf, 1% denormals, 1% +-0 and the rest
    normal(0, 1e3); candidate flips the sign of zeros and changes NaN payloads
    with probability 1/2 each; equal_nan true, rtol 1e-7, atol 0."""
    ref = TensorSpec(n, "f32", "special",
                     dict(mean=0.0, std=1e3, p_nan=0.01, p_inf=0.005, p_denorm=0.01, p_zero=0.01))
    steps = [Step("special_flip", p=0.5, stream=harness_stream(TAG_FLIP, 0))]
    return Workload("special_f32_%d" % n, [Case(ref, steps, 1e-7, 0.0, True)], False,
                    "%d fp32 special mix; zero sign flips + NaN payload changes" % n,
                    expect=dict(mismatches=0, err_sum=0.0))


def candidates_round(outputs: int = 8, n: int = 1 << 24, G: int = 3) -> Workload:
    """One round of the generation loop (Sec. 5.1: G = 3 kernels per round)
    validated in one batched check: 8 outputs of 2^24 fp32 normal(5, 10)
    (streams 0..7), each checked against 3 candidates -- the first reproduces
    the reference, the second is off everywhere (x(1+u), |u| <= 1e-2), the
    third has one wrong element at a seeded index; rtol 1e-5, atol 1e-6.  The
    check stops each failing segment at its first mismatch (fail-fast,
    Sec. 4.2.2)."""
    rng = np.random.Generator(np.random.PCG64(1006))
    cases, faults = [], {}
    for j in range(outputs):
        ref = TensorSpec(n, "f32", "normal", dict(mean=5.0, std=10.0), stream=j)
        for g in range(G):
            if g % 3 == 0:
                steps = [Step("copy")]
            elif g % 3 == 1:
                steps = [Step("scale", p=1.0, value=1e-2, stream=harness_stream(TAG_SCALE, 1000 + G * j + g))]
            else:
                pos = np.array([rng.integers(0, n)], dtype=np.uint64)
                faults[len(cases)] = int(pos[0])
                steps = [Step("copy"), Step("fault_at", idx=pos)]
            cases.append(Case(ref, steps, 1e-5, 1e-6, False))
    return Workload("candidates_round_%dx%dx%d" % (outputs, G, n), cases, True,
                    "%d fp32 outputs of %d elements x %d candidates (exact, off everywhere, one fault); "
                    "stop at first mismatch" % (outputs, n, G),
                    expect=dict(faults=faults), stop_at_first=True)


WORKLOADS = {
    "uniform_small": uniform_small,
    "normal_ulp": normal_ulp,
    "bf16_batch": bf16_batch,
    "ragged_batch": ragged_batch,
    "special_stream": special_stream,
    "candidates_round": candidates_round,
}

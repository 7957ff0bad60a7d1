"""Kernel timing of the library's own launches (sv_profile_enable /
sv_profile_read), which the benchmark's per-kernel figures and roofline rest
on: every launch of a kind is counted once, durations are positive and fit
inside the wall time of the calls that made them, reads forget what they
returned, and nothing is recorded while timing is off."""
import numpy as np
import pytest
import torch

import paper_2609_00058_amd as sv
from gpu_run import empty

pytestmark = pytest.mark.gpu

KINDS = ("synth", "compare", "perturb", "finalize")


def test_launches_are_counted_and_timed():
    big = empty(1 << 24, "f32")
    cand = torch.empty_like(big)
    small = empty(1000, "f32")
    sv.synth(small, 0, 0, "uniform", a=0.0, b=1.0)
    torch.cuda.synchronize()
    for k in KINDS:
        sv.profile_read(k)                                   # forget anything recorded before
    sv.profile_enable(True)
    try:
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for s in range(3):
            sv.synth(big, s, 1, "normal", mean=0.0, std=1.0)
        b.record()
        sv.perturb(big, cand, 7, 8, "ulp", p=0.01)
        for _ in range(2):
            sv.compare(big, cand, 1e-6, 0.0)                 # a full grid: check kernel + finalize kernel
        sv.compare(small, small, 0.0, 0.0)                   # one workgroup reports by itself: no finalize
        b.synchronize()
        wall_synth = a.elapsed_time(b)
        got = {k: sv.profile_read(k) for k in KINDS}
    finally:
        sv.profile_enable(False)
    assert got["synth"][0] == 3 and got["perturb"][0] == 1
    assert got["compare"][0] == 3 and got["finalize"][0] == 2
    for k in KINDS:
        assert got[k][1] > 0.0, k
    assert got["synth"][1] <= wall_synth * 1.05 + 0.05, (got["synth"], wall_synth)
    # read again: forgotten; launches while off: not recorded
    assert all(sv.profile_read(k) == (0, 0.0) for k in KINDS)
    sv.synth(big, 9, 1, "normal", mean=0.0, std=1.0)
    sv.compare(big, big, 0.0, 0.0)
    torch.cuda.synchronize()
    assert all(sv.profile_read(k)[0] == 0 for k in KINDS)

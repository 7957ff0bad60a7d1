"""sv_shutdown frees every scratch area; later calls allocate again and give
the same results.  A check still pending at the shutdown is forgotten: waiting
for its ticket afterwards is an error, not a hang or a crash."""
import numpy as np
import pytest
import torch

import paper_2609_00058_amd as sv
from gpu_run import bits, empty, same_report

pytestmark = pytest.mark.gpu


def _work(tmp_path, tag):
    ref = empty((1 << 22) + 5, "f32")
    sv.synth(ref, 1, 2, "special", mean=0.0, std=100.0, p_nan=0.01, p_inf=0.01, p_denorm=0.01, p_zero=0.01)
    cand = torch.empty_like(ref)
    sv.perturb(ref, cand, 3, 4, "ulp", p=0.01)
    sv.perturb(ref, cand, 3, 5, "fault_at", idx=np.array([7, 1 << 21], dtype=np.uint64))
    small = empty(1000, "bf16")
    sv.synth_batched([(small, 5, 6, "uniform", dict(a=-1.0, b=1.0)), (empty(7, "i32"), 1, 1, "int_range",
                                                                      dict(lo=0, hi=9))])
    segs = [(ref, cand, 1e-6, 0.0, True), (small, small, 0.0, 0.0, False), (ref[:100], cand[:100], 0.0, 0.0, False)]
    path = str(tmp_path / ("ref_%s.bin" % tag))
    sv.synth_file(path, 10000, 1, 2, "f32", "normal", mean=0.0, std=1.0)
    return dict(single=sv.compare(ref, cand, 1e-6, 0.0, True), noalloc=sv.compare_noalloc(ref, cand, 1e-6, 0.0, True),
                batched=sv.compare_batched(segs), stop=sv.compare_batched(segs, stop_at_first=True),
                submitted=sv.compare_submit(ref, cand, 1e-6, 0.0, True).wait(),
                ref=bits(ref), small=bits(small), file=sv.compare_file(path, path, 10000, "f32", 0.0, 0.0))


def test_shutdown_then_everything_again(tmp_path):
    before = _work(tmp_path, "a")
    ref = empty(1 << 20, "f32")
    sv.synth(ref, 9, 9, "normal", mean=0.0, std=1.0)
    pending = sv.compare_submit(ref, ref, 0.0, 0.0)            # left pending across the shutdown
    sv.shutdown()
    with pytest.raises(sv.SVError):
        pending.wait()
    sv.shutdown()                                              # twice in a row: nothing left to free
    after = _work(tmp_path, "b")
    for k in ("single", "noalloc", "submitted", "file"):
        same_report(after[k], before[k])
    for k in ("batched", "stop"):
        for g, w in zip(after[k], before[k]):
            same_report(g, w)
    assert np.array_equal(after["ref"], before["ref"]) and np.array_equal(after["small"], before["small"])
    assert sv.compare_submit(ref, ref, 0.0, 0.0).wait()["mismatches"] == 0

"""Run a workload case through libsynthverify on the GPU (test helper)."""
import numpy as np
import torch

import paper_2609_00058_amd as sv

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16, "i32": torch.int32, "f16": torch.float16,
               "f64": torch.float64, "u8": torch.uint8, "i64": torch.int64}
STORAGE = {"f32": np.uint32, "bf16": np.uint16, "i32": np.uint32, "f16": np.uint16, "f64": np.uint64,
           "u8": np.uint8, "i64": np.uint64}


def empty(n, dtype, device="cuda"):
    return torch.empty(n, dtype=TORCH_DTYPE[dtype], device=device)


def gpu_ref(spec, out=None):
    out = empty(spec.n, spec.dtype) if out is None else out
    sv.synth(out, spec.seed, spec.stream, spec.dist, **spec.params)
    return out


def gpu_cand(case, ref, cand=None):
    cand = torch.empty_like(ref) if cand is None else cand
    for s in case.steps:
        if s.op in ("copy", "ulp", "scale", "special_flip"):
            sv.perturb(ref, cand, s.seed, s.stream, s.op, p=s.p, value=s.value)
        else:
            sv.perturb(ref, cand, s.seed, s.stream, s.op, value=s.value, bits=s.bits, idx=s.idx)
    return cand


def bits(t):
    """Raw storage of a device tensor as a host numpy array."""
    if t.dtype in (torch.bfloat16, torch.float16):
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    if t.dtype == torch.uint8:
        return t.cpu().numpy()
    if t.dtype in (torch.float64, torch.int64):
        return t.view(torch.int64).cpu().numpy().view(np.uint64)
    return t.view(torch.int32).cpu().numpy().view(np.uint32)


def dev_bits(arr, dtype):
    """A device tensor of `dtype` holding the raw storage array `arr`."""
    view = {np.uint16: np.int16, np.uint32: np.int32, np.uint64: np.int64, np.uint8: np.uint8}
    a = np.ascontiguousarray(arr)
    t = torch.from_numpy(a.view(view[a.dtype.type])).to("cuda")
    return t.view(TORCH_DTYPE[dtype])


def bits_at(t, idx):
    ii = torch.as_tensor(np.asarray(idx, dtype=np.int64), device=t.device)
    return bits(t.index_select(0, ii))


def same_report(got, want, sum_rel=1e-12):
    """Bit-exact on every field except err_sum (within sum_rel relative; an
    exact 0 or an overflow to +Inf must match exactly)."""
    for k in want:
        if k == "err_sum":
            if want[k] == 0.0 or want[k] == float("inf"):
                assert got[k] == want[k], (k, got[k], want[k])
            else:
                assert abs(got[k] - want[k]) <= sum_rel * abs(want[k]), (k, got[k], want[k])
        else:
            assert got[k] == want[k], (k, got[k], want[k])

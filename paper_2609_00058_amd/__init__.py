"""Python binding of libsynthverify (argument marshalling only).

Seeded synthesis of test inputs and the elementwise check of Eq. (1) of
"CUDA-Harness" (arXiv 2609.00058, Sec. 4.2) on an MI355X.  Every step runs in
the HIP kernels of libsynthverify.so; this module turns torch tensors into
device pointers, passes torch's current HIP stream to the library, and
returns reports as dicts.  It never computes anything itself and has no CPU
fallback: if the library is missing, importing this package fails.
"""
import ctypes
import os
import threading

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsynthverify.so")

if not os.path.exists(LIB_PATH):
    raise ImportError("libsynthverify.so is not built (run paper_2609_00058_amd/build.py or "
                      "__graft_entry__.build())")

# torch first: the library must run on the HIP runtime that torch loads (its
# own libamdhip64.so.7), which the library's dependency of the same name then
# binds to.  Loaded before torch, the library would bring in the system's copy,
# and the process would hold two HIP runtimes, of which the library's finds no
# device (measured: "no ROCm-capable device is detected" on every call).
import torch  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)

SV_OK, SV_ERR_INVALID_ARG, SV_ERR_UNSUPPORTED, SV_ERR_HIP, SV_ERR_ALLOC, SV_ERR_IO = 0, -1, -2, -3, -4, -5
SV_MAX_PENDING_CHECKS = 16   # submitted checks per device not yet waited for
DTYPE_CODES = {"f32": 0, "bf16": 1, "i32": 2, "f16": 3, "f64": 4, "u8": 5, "i64": 6}
DIST_CODES = {"uniform": 0, "normal": 1, "int_range": 2, "special": 3, "permutation": 4}
OP_CODES = {"copy": 0, "ulp": 1, "scale": 2, "special_flip": 3,
            "add_at": 4, "set_at": 5, "fault_at": 6}
PROF_KINDS = {"synth": 0, "compare": 1, "perturb": 2, "finalize": 3}

# every symbol include/sv.h declares
SYMBOLS = ("sv_synth", "sv_synth_batched", "sv_synth_window", "sv_compare", "sv_compare_batched", "sv_compare_batched_mode",
           "sv_compare_submit", "sv_compare_batched_submit", "sv_compare_ready", "sv_compare_wait", "sv_perturb",
           "sv_eval_transform", "sv_synth_file", "sv_compare_file", "sv_kernel_load", "sv_kernel_free", "sv_kernel_launch", "sv_kernel_time",
           "sv_reward", "sv_set_stream", "sv_last_error", "sv_profile_enable", "sv_profile_read", "sv_shutdown",
           "sv_testing_set_sequence", "sv_abi_version", "sv_compare_noalloc")


class DistParams(ctypes.Structure):
    _fields_ = [("a", ctypes.c_double), ("b", ctypes.c_double),
                ("mean", ctypes.c_double), ("std", ctypes.c_double),
                ("lo", ctypes.c_int64), ("hi", ctypes.c_int64),
                ("p_nan", ctypes.c_double), ("p_inf", ctypes.c_double),
                ("p_denorm", ctypes.c_double), ("p_zero", ctypes.c_double)]


class SynthJob(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("stream_id", ctypes.c_uint64),
                ("dtype", ctypes.c_int32), ("dist", ctypes.c_int32),
                ("params", DistParams), ("n", ctypes.c_uint64), ("out", ctypes.c_void_p)]


class Report(ctypes.Structure):
    _fields_ = [("n", ctypes.c_uint64), ("mismatches", ctypes.c_uint64),
                ("first_mismatch", ctypes.c_int64),
                ("max_abs_err", ctypes.c_double), ("max_rel_err", ctypes.c_double),
                ("err_sum", ctypes.c_double),
                ("nan_ref", ctypes.c_uint64), ("nan_cand", ctypes.c_uint64),
                ("inf_ref", ctypes.c_uint64), ("inf_cand", ctypes.c_uint64)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


# the same layout as a numpy structured type: reports as one array, without a
# Python object per report (as_array=True below)
REPORT_DTYPE = np.dtype([(name, {ctypes.c_uint64: "<u8", ctypes.c_int64: "<i8", ctypes.c_double: "<f8"}[t])
                         for name, t in Report._fields_])
assert REPORT_DTYPE.itemsize == ctypes.sizeof(Report)


def _reports(reps, n: int, as_array: bool):
    if as_array:
        return np.frombuffer(reps, dtype=REPORT_DTYPE, count=n)   # a view of the filled array
    return [reps[k].as_dict() for k in range(n)]


class Segment(ctypes.Structure):
    _fields_ = [("ref", ctypes.c_void_p), ("cand", ctypes.c_void_p),
                ("n", ctypes.c_uint64), ("dtype", ctypes.c_int32),
                ("rtol", ctypes.c_double), ("atol", ctypes.c_double),
                ("equal_nan", ctypes.c_int32)]


class PerturbPlan(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("p", ctypes.c_double),
                ("value", ctypes.c_double), ("bits", ctypes.c_uint32),
                ("idx", ctypes.POINTER(ctypes.c_uint64)), ("nidx", ctypes.c_uint64)]


class Launch(ctypes.Structure):
    _fields_ = [("grid", ctypes.c_uint32 * 3), ("block", ctypes.c_uint32 * 3),
                ("shared_bytes", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("args", ctypes.c_void_p), ("args_size", ctypes.c_uint64)]


class Timing(ctypes.Structure):
    _fields_ = [("reps", ctypes.c_uint32), ("reserved", ctypes.c_uint32),
                ("mean_ms", ctypes.c_double), ("median_ms", ctypes.c_double),
                ("min_ms", ctypes.c_double), ("max_ms", ctypes.c_double), ("perf", ctypes.c_double)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_ if name != "reserved"}


_u64, _i32, _vp, _dbl = ctypes.c_uint64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_double
_lib.sv_synth.argtypes = [_u64, _u64, _i32, _i32, ctypes.POINTER(DistParams), _u64, _vp]
_lib.sv_synth_batched.argtypes = [ctypes.POINTER(SynthJob), ctypes.c_uint32]
_lib.sv_synth_window.argtypes = [_u64, _u64, _i32, _i32, ctypes.POINTER(DistParams), _u64, _u64, _vp]
_lib.sv_compare.argtypes = [_vp, _vp, _u64, _i32, _dbl, _dbl, _i32, ctypes.POINTER(Report)]
_lib.sv_compare_noalloc.argtypes = [_vp, _vp, _u64, _i32, _dbl, _dbl, _i32, ctypes.POINTER(Report)]
_lib.sv_compare_batched.argtypes = [ctypes.POINTER(Segment), ctypes.c_uint32, ctypes.POINTER(Report)]
_lib.sv_compare_batched_mode.argtypes = [ctypes.POINTER(Segment), ctypes.c_uint32, _i32, ctypes.POINTER(Report)]
_lib.sv_compare_submit.argtypes = [_vp, _vp, _u64, _i32, _dbl, _dbl, _i32, ctypes.POINTER(_u64)]
_lib.sv_compare_batched_submit.argtypes = [ctypes.POINTER(Segment), ctypes.c_uint32, _i32, ctypes.POINTER(_u64)]
_lib.sv_compare_ready.argtypes = [_u64, ctypes.POINTER(_i32)]
_lib.sv_compare_wait.argtypes = [_u64, ctypes.POINTER(Report), ctypes.c_uint32]
_lib.sv_perturb.argtypes = [_u64, _u64, _i32, ctypes.POINTER(PerturbPlan), _u64, _vp, _vp]
_lib.sv_eval_transform.argtypes = [_i32, _vp, _u64, _vp]
_lib.sv_kernel_load.argtypes = [ctypes.c_char_p, _u64, ctypes.c_char_p, ctypes.POINTER(_vp)]
_lib.sv_kernel_free.argtypes = [_vp]
_lib.sv_kernel_launch.argtypes = [_vp, ctypes.POINTER(Launch)]
_lib.sv_kernel_time.argtypes = [_vp, ctypes.POINTER(Launch), ctypes.c_uint32, ctypes.c_uint32, _u64,
                                ctypes.POINTER(ctypes.c_float), ctypes.POINTER(Timing)]
_lib.sv_synth_file.argtypes = [ctypes.c_char_p, _u64, _u64, _i32, _i32, ctypes.POINTER(DistParams), _u64]
_lib.sv_compare_file.argtypes = [ctypes.c_char_p, ctypes.c_char_p, _u64, _i32, _dbl, _dbl, _i32,
                                 ctypes.POINTER(Report)]
_lib.sv_set_stream.argtypes = [_vp]
_lib.sv_testing_set_sequence.argtypes = [_u64]
_lib.sv_last_error.restype = ctypes.c_char_p
_lib.sv_profile_enable.argtypes = [_i32]
_lib.sv_profile_read.argtypes = [_i32, ctypes.POINTER(_u64), ctypes.POINTER(_dbl)]
for _name in SYMBOLS:
    if _name not in ("sv_last_error", "sv_reward"):
        getattr(_lib, _name).restype = ctypes.c_int
_lib.sv_reward.argtypes = [_i32, _i32, _dbl]
_lib.sv_reward.restype = _dbl


class SVError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("libsynthverify error %d: %s" % (code, msg))
        self.code = code


def _check(rc):
    if rc != SV_OK:
        raise SVError(rc, _lib.sv_last_error().decode(errors="replace"))


def lib():
    return _lib


_torch_mod = None
_tdtype_codes = None
_tls = threading.local()


def _torch():
    global _torch_mod, _tdtype_codes
    if _torch_mod is None:
        import torch
        _torch_mod = torch
        _tdtype_codes = {torch.float32: 0, torch.bfloat16: 1, torch.int32: 2, torch.float16: 3,
                         torch.float64: 4, torch.uint8: 5, torch.int64: 6}
    return _torch_mod


def dtype_code(t) -> int:
    _torch()
    code = _tdtype_codes.get(t.dtype)
    if code is None:
        raise SVError(SV_ERR_UNSUPPORTED, "unsupported tensor dtype %s" % t.dtype)
    return code


def _dev_ptr(t, name):
    if not t.is_cuda:
        raise SVError(SV_ERR_INVALID_ARG, "%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise SVError(SV_ERR_INVALID_ARG, "%s must be contiguous" % name)
    return t.data_ptr()


def _run(t, fn, *args):
    """Call fn(*args) with t's device current and torch's current stream of
    that device handed to the library (only when it changed)."""
    dev = t.get_device()
    if dev < 0:
        raise SVError(SV_ERR_INVALID_ARG, "tensors must be on the GPU")
    _run_on(dev, fn, *args)


def _run_on(dev, fn, *args):
    torch = _torch()
    prev = torch._C._cuda_getDevice()
    if prev != dev:
        torch.cuda.set_device(dev)
    try:
        stream = torch._C._cuda_getCurrentRawStream(dev)
        if getattr(_tls, "stream", None) != (dev, stream):
            _check(_lib.sv_set_stream(stream))
            _tls.stream = (dev, stream)
        _check(fn(*args))
    finally:
        if prev != dev:
            torch.cuda.set_device(prev)


def dist_params(**kw) -> DistParams:
    p = DistParams()
    for k, v in kw.items():
        setattr(p, k, v)
    return p


def synth(out, seed: int, stream_id: int, dist: str, **params):
    """Fill `out` (contiguous device tensor) with the seeded sequence (asynchronous)."""
    _run(out, _lib.sv_synth, seed, stream_id, dtype_code(out), DIST_CODES[dist],
         ctypes.byref(dist_params(**params)), out.numel(), _dev_ptr(out, "out"))
    return out


def synth_window(out, seed: int, stream_id: int, dist: str, offset: int, **params):
    """Fill `out` with elements [offset, offset + out.numel()) of the tensor synth() would produce."""
    p = dist_params(**params)
    _run(out, _lib.sv_synth_window, seed, stream_id, dtype_code(out), DIST_CODES[dist], ctypes.byref(p), offset,
         out.numel(), _dev_ptr(out, "out"))
    return out


def _run_current(fn, *args):
    torch = _torch()
    _run_on(torch._C._cuda_getDevice(), fn, *args)


def synth_file(path: str, n: int, seed: int, stream_id: int, dtype: str, dist: str, **params):
    """Write the n elements synth() would produce, raw, to `path` (on the current device; synchronous)."""
    _run_current(_lib.sv_synth_file, os.fsencode(path), seed, stream_id, DTYPE_CODES[dtype], DIST_CODES[dist],
                 ctypes.byref(dist_params(**params)), n)


def compare_file(ref_path: str, cand_path: str, n: int, dtype: str, rtol: float, atol: float,
                 equal_nan: bool = False) -> dict:
    """Eq. (1) between two raw files of n elements of `dtype` (on the current device)."""
    r = Report()
    _run_current(_lib.sv_compare_file, os.fsencode(ref_path), os.fsencode(cand_path), n, DTYPE_CODES[dtype],
                 rtol, atol, int(bool(equal_nan)), ctypes.byref(r))
    return r.as_dict()


class SynthBatch:
    """The jobs of synth_batched() marshalled once, for a batch synthesized
    again and again: pass it to synth_batched() in place of the list.  It
    keeps its output tensors alive."""

    def __init__(self, jobs):
        if not jobs:
            raise SVError(SV_ERR_INVALID_ARG, "SynthBatch: no jobs")
        self.arr = (SynthJob * len(jobs))()
        for k, (out, seed, stream_id, dist, params) in enumerate(jobs):
            self.arr[k] = SynthJob(seed, stream_id, dtype_code(out), DIST_CODES[dist], dist_params(**params),
                                   out.numel(), _dev_ptr(out, "out") if out.numel() else None)
        self.n = len(jobs)
        self.outs = [j[0] for j in jobs]


def synth_batched(jobs):
    """jobs: list of (out, seed, stream_id, dist, params dict), or a SynthBatch;
    one launch (asynchronous)."""
    if not isinstance(jobs, SynthBatch):
        if not jobs:
            return
        jobs = SynthBatch(jobs)
    _run(jobs.outs[0], _lib.sv_synth_batched, jobs.arr, jobs.n)


def compare(ref, cand, rtol: float, atol: float, equal_nan: bool = False) -> dict:
    """Eq. (1) on every element of (ref, cand) -> report dict (synchronous)."""
    if ref.dtype != cand.dtype or ref.numel() != cand.numel():
        raise SVError(SV_ERR_INVALID_ARG, "ref and cand must have the same dtype and size")
    rep = Report()
    _run(ref, _lib.sv_compare, _dev_ptr(ref, "ref"), _dev_ptr(cand, "cand"), ref.numel(), dtype_code(ref),
         rtol, atol, int(bool(equal_nan)), ctypes.byref(rep))
    return rep.as_dict()


def compare_noalloc(ref, cand, rtol: float, atol: float, equal_nan: bool = False) -> dict:
    """compare() through sv_compare_noalloc: the library's fixed device scratch,
    nothing allocated (synchronous)."""
    if ref.dtype != cand.dtype or ref.numel() != cand.numel():
        raise SVError(SV_ERR_INVALID_ARG, "ref and cand must have the same dtype and size")
    rep = Report()
    _run(ref, _lib.sv_compare_noalloc, _dev_ptr(ref, "ref"), _dev_ptr(cand, "cand"), ref.numel(), dtype_code(ref),
         rtol, atol, int(bool(equal_nan)), ctypes.byref(rep))
    return rep.as_dict()


def _segment_array(segments):
    arr = (Segment * len(segments))()
    for k, (ref, cand, rtol, atol, eqn) in enumerate(segments):
        if ref.dtype != cand.dtype or ref.numel() != cand.numel():
            raise SVError(SV_ERR_INVALID_ARG, "segment %d: ref and cand differ in dtype or size" % k)
        arr[k] = Segment(_dev_ptr(ref, "ref") if ref.numel() else None,
                         _dev_ptr(cand, "cand") if cand.numel() else None,
                         ref.numel(), dtype_code(ref), rtol, atol, int(bool(eqn)))
    return arr


class SegmentBatch:
    """The segments of compare_batched() marshalled once, for a batch checked
    again and again: pass it in place of the list to compare_batched() or
    compare_batched_submit().  It keeps its tensors alive."""

    def __init__(self, segments):
        if not segments:
            raise SVError(SV_ERR_INVALID_ARG, "SegmentBatch: no segments")
        self.arr = _segment_array(segments)
        self.n = len(segments)
        self.tensors = [s[:2] for s in segments]


def _as_batch(segments):
    return segments if isinstance(segments, SegmentBatch) else SegmentBatch(segments)


def compare_batched(segments, stop_at_first: bool = False, as_array: bool = False):
    """segments: list of (ref, cand, rtol, atol, equal_nan), or a SegmentBatch;
    one launch, one report each (a list of dicts, or with as_array a numpy array
    of REPORT_DTYPE, one record per segment).
    stop_at_first: a failing segment is checked only as far as needed to know
    its first mismatch exactly; its report then holds n, mismatches = 1 and
    first_mismatch, everything else 0."""
    if not isinstance(segments, SegmentBatch) and not segments:
        return np.zeros(0, REPORT_DTYPE) if as_array else []
    b = _as_batch(segments)
    reps = (Report * b.n)()
    _run(b.tensors[0][0], _lib.sv_compare_batched_mode, b.arr, b.n, 1 if stop_at_first else 0, reps)
    return _reports(reps, b.n, as_array)


class CheckTicket:
    """A submitted check (compare_submit, compare_batched_submit).  It keeps its
    tensors alive until waited for; wait() returns what compare() or
    compare_batched() would have returned (with as_array, the reports as a numpy
    array of REPORT_DTYPE, one record per segment, also for a single tensor).
    The check's last reduction step may be left to the next check submitted on
    the same stream; ready() and wait() queue it themselves when none comes, so
    poll ready() (or wait) rather than relying on a stream synchronization."""

    def __init__(self, ticket: int, nreports: int, batched: bool, keep):
        self.ticket, self.nreports, self.batched, self._keep = ticket, nreports, batched, keep
        self._reps, self._result = None, None

    def ready(self) -> bool:
        if self._reps is not None:
            return True
        flag = ctypes.c_int32(0)
        _check(_lib.sv_compare_ready(self.ticket, ctypes.byref(flag)))
        return bool(flag.value)

    def wait(self, as_array: bool = False):
        if self._reps is None:
            reps = (Report * max(self.nreports, 1))()
            _check(_lib.sv_compare_wait(self.ticket, reps, self.nreports))
            self._reps, self._keep = reps, None
        if as_array:
            return _reports(self._reps, self.nreports, True)
        if self._result is None:
            out = _reports(self._reps, self.nreports, False)
            self._result = out if self.batched else out[0]
        return self._result


def compare_submit(ref, cand, rtol: float, atol: float, equal_nan: bool = False) -> CheckTicket:
    """compare() queued on the current stream without waiting; .wait() gives the report."""
    if ref.dtype != cand.dtype or ref.numel() != cand.numel():
        raise SVError(SV_ERR_INVALID_ARG, "ref and cand must have the same dtype and size")
    t = ctypes.c_uint64(0)
    _run(ref, _lib.sv_compare_submit, _dev_ptr(ref, "ref"), _dev_ptr(cand, "cand"), ref.numel(),
         dtype_code(ref), rtol, atol, int(bool(equal_nan)), ctypes.byref(t))
    return CheckTicket(t.value, 1, False, (ref, cand))


def compare_batched_submit(segments, stop_at_first: bool = False) -> CheckTicket:
    """compare_batched() queued on the current stream without waiting; .wait() gives the reports."""
    if not isinstance(segments, SegmentBatch) and not segments:
        raise SVError(SV_ERR_INVALID_ARG, "compare_batched_submit: no segments")
    b = _as_batch(segments)
    t = ctypes.c_uint64(0)
    _run(b.tensors[0][0], _lib.sv_compare_batched_submit, b.arr, b.n, 1 if stop_at_first else 0, ctypes.byref(t))
    return CheckTicket(t.value, b.n, True, b)


class _Prepared:
    """A library call with its arguments marshalled once, for calls repeated on
    the same tensors: each call hands torch's current stream of the device to
    the library (when it changed) and calls it.  Keeps its tensors alive."""

    def __init__(self, dev, keep):
        self._dev = dev
        self._keep = keep

    def _call(self, fn, *args):
        torch = _torch()
        dev = self._dev
        if torch._C._cuda_getDevice() != dev:
            return _run_on(dev, fn, *args)
        stream = torch._C._cuda_getCurrentRawStream(dev)
        if getattr(_tls, "stream", None) != (dev, stream):
            _check(_lib.sv_set_stream(stream))
            _tls.stream = (dev, stream)
        rc = fn(*args)
        if rc:
            _check(rc)


class PreparedSynth(_Prepared):
    """synth(out, seed, stream_id, dist, **params) marshalled once; call it to launch."""

    def __init__(self, out, seed: int, stream_id: int, dist: str, **params):
        super().__init__(out.get_device(), out)
        self._params = dist_params(**params)
        self._args = (ctypes.c_uint64(seed), ctypes.c_uint64(stream_id), ctypes.c_int32(dtype_code(out)),
                      ctypes.c_int32(DIST_CODES[dist]), ctypes.byref(self._params), ctypes.c_uint64(out.numel()),
                      ctypes.c_void_p(_dev_ptr(out, "out") if out.numel() else None))

    def __call__(self):
        self._call(_lib.sv_synth, *self._args)


class PreparedCheck(_Prepared):
    """compare(ref, cand, rtol, atol, equal_nan) marshalled once: run() checks and
    returns the report, submit() queues the check and returns its ticket."""

    def __init__(self, ref, cand, rtol: float, atol: float, equal_nan: bool = False):
        if ref.dtype != cand.dtype or ref.numel() != cand.numel():
            raise SVError(SV_ERR_INVALID_ARG, "ref and cand must have the same dtype and size")
        super().__init__(ref.get_device(), (ref, cand))
        n = ref.numel()
        self._args = (ctypes.c_void_p(_dev_ptr(ref, "ref") if n else None),
                      ctypes.c_void_p(_dev_ptr(cand, "cand") if n else None), ctypes.c_uint64(n),
                      ctypes.c_int32(dtype_code(ref)), ctypes.c_double(rtol), ctypes.c_double(atol),
                      ctypes.c_int32(int(bool(equal_nan))))
        self._rep = Report()
        self._ticket = ctypes.c_uint64(0)

    def run(self) -> dict:
        self._call(_lib.sv_compare, *self._args, ctypes.byref(self._rep))
        return self._rep.as_dict()

    def submit(self) -> CheckTicket:
        self._call(_lib.sv_compare_submit, *self._args, ctypes.byref(self._ticket))
        return CheckTicket(self._ticket.value, 1, False, self)


def perturb(ref, cand, seed: int, stream_id: int, op: str, p: float = 0.0, value: float = 0.0,
            bits: int = 0, idx=None):
    """One candidate-derivation step from ref into cand (workload support)."""
    import numpy as np
    if ref.dtype != cand.dtype or ref.numel() != cand.numel():
        raise SVError(SV_ERR_INVALID_ARG, "ref and cand must have the same dtype and size")
    idx_arr = np.ascontiguousarray(idx if idx is not None else [], dtype=np.uint64)
    plan = PerturbPlan(OP_CODES[op], p, value, bits & 0xFFFFFFFF,
                       idx_arr.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)), idx_arr.size)
    _run(ref, _lib.sv_perturb, seed, stream_id, dtype_code(ref), ctypes.byref(plan), ref.numel(),
         _dev_ptr(ref, "ref"), _dev_ptr(cand, "cand"))
    return cand


EVAL = {"ln": 0, "radius": 1, "sin": 2, "cos": 3, "f16": 4, "bf16": 5}


def eval_transform(which: str, inp, out):
    """Diagnostics: one building block of the normal transform on int32 device tensors (asynchronous)."""
    if inp.numel() != out.numel():
        raise SVError(SV_ERR_INVALID_ARG, "in and out differ in size")
    _run(inp, _lib.sv_eval_transform, EVAL[which], _dev_ptr(inp, "in"), inp.numel(), _dev_ptr(out, "out"))
    return out


class Kernel:
    """A candidate kernel loaded from a gfx950 code object (sv_kernel_load)."""

    def __init__(self, code_object: bytes, name: str, device: int = None):
        torch = _torch()
        self.device = torch._C._cuda_getDevice() if device is None else device
        self._code = bytes(code_object)
        self.name = name
        h = _vp()
        _run_on(self.device, _lib.sv_kernel_load, self._code, len(self._code), name.encode(), ctypes.byref(h))
        self._h = h

    def free(self):
        if getattr(self, "_h", None):
            _check(_lib.sv_kernel_free(self._h))
            self._h = None

    def _launch_struct(self, grid, block, args, shared_bytes):
        grid = tuple(grid) + (1,) * (3 - len(grid))
        block = tuple(block) + (1,) * (3 - len(block))
        buf = ctypes.create_string_buffer(bytes(args), len(args)) if args else None
        l = Launch((ctypes.c_uint32 * 3)(*grid), (ctypes.c_uint32 * 3)(*block), shared_bytes, 0,
                   ctypes.cast(buf, _vp) if buf is not None else None, len(args) if args else 0)
        return l, buf

    def launch(self, grid, block, args: bytes = b"", shared_bytes: int = 0):
        """One launch on torch's current stream (asynchronous)."""
        l, buf = self._launch_struct(grid, block, args, shared_bytes)
        _run_on(self.device, _lib.sv_kernel_launch, self._h, ctypes.byref(l))

    def time(self, grid, block, args: bytes = b"", shared_bytes: int = 0, warmup: int = 3, reps: int = 20,
             flush_bytes: int = 0, per_rep: bool = False) -> dict:
        """The performance stage: latency statistics and P = 1 / mean latency (1/ms)."""
        l, buf = self._launch_struct(grid, block, args, shared_bytes)
        out = Timing()
        arr = (ctypes.c_float * reps)() if per_rep else None
        _run_on(self.device, _lib.sv_kernel_time, self._h, ctypes.byref(l), warmup, reps, flush_bytes, arr,
                ctypes.byref(out))
        d = out.as_dict()
        if per_rep:
            d["rep_ms"] = list(arr)
        return d

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def kernel_load(code_object: bytes, name: str) -> Kernel:
    return Kernel(code_object, name)


def reward(compiled: bool, valid: bool, perf: float) -> float:
    """Eq. (4): r = -1 + C + C V P."""
    return _lib.sv_reward(1 if compiled else 0, 1 if valid else 0, float(perf))


def profile_enable(on: bool = True):
    _check(_lib.sv_profile_enable(int(bool(on))))


def profile_read(kind: str):
    """(count, total_ms) of the main-kernel events of `kind` recorded since the last read."""
    c, ms = ctypes.c_uint64(), ctypes.c_double()
    _check(_lib.sv_profile_read(PROF_KINDS[kind], ctypes.byref(c), ctypes.byref(ms)))
    return c.value, ms.value


def shutdown():
    _check(_lib.sv_shutdown())

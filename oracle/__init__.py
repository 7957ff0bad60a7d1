"""CPU test oracle for seeded synthesis and the elementwise check of Eq. (1).

TEST INFRASTRUCTURE ONLY: tests, the smoke entry and the benchmark's CPU
baseline leg may use this package; the product path never does, and this
package imports nothing from the product.  It wraps the plain serial C in
sv_oracle.c (numpy arrays in, numpy arrays out) using the oracle's own enum
values; callers name dtypes, distributions and ops by string.

Parity status of each function (what pins it is in tests/test_oracle_*.py):
  philox            pinned: Random123 known-answer vectors, rocRAND run on host
  synth uniform     pinned: closed form on power-of-two spans, moments, KS
  synth normal      pinned: per-element error vs float64 Box-Muller, moments, KS
  synth int_range   pinned: closed form on power-of-two ranges, bounds, chi^2
  synth special     pinned: class frequencies, bit-pattern rules, KS of normals
  bf16 rounding     pinned: torch CPU float32 -> bfloat16 conversion
  perturb           pinned: numpy.nextafter, brute-force bf16 order, exact
                    rational arithmetic of the scale op
  compare           pinned: exact rational evaluation of Eq. (1), numpy.isclose,
                    math.fsum, numpy max
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsvoracle.so")

DTYPES = {"f32": 0, "bf16": 1, "i32": 2, "f16": 3, "f64": 4, "u8": 5, "i64": 6}
NP_STORAGE = {"f32": np.uint32, "bf16": np.uint16, "i32": np.uint32, "f16": np.uint16, "f64": np.uint64,
              "u8": np.uint8, "i64": np.uint64}
DISTS = {"uniform": 0, "normal": 1, "int_range": 2, "special": 3, "permutation": 4}
OPS = {"copy": 0, "ulp": 1, "scale": 2, "special_flip": 3,
       "add_at": 4, "set_at": 5, "fault_at": 6}


class DistParams(ctypes.Structure):
    _fields_ = [("a", ctypes.c_double), ("b", ctypes.c_double),
                ("mean", ctypes.c_double), ("std", ctypes.c_double),
                ("lo", ctypes.c_int64), ("hi", ctypes.c_int64),
                ("p_nan", ctypes.c_double), ("p_inf", ctypes.c_double),
                ("p_denorm", ctypes.c_double), ("p_zero", ctypes.c_double)]


class PerturbPlan(ctypes.Structure):
    _fields_ = [("op", ctypes.c_int32), ("p", ctypes.c_double),
                ("value", ctypes.c_double), ("bits", ctypes.c_uint32),
                ("idx", ctypes.POINTER(ctypes.c_uint64)), ("nidx", ctypes.c_uint64)]


class Report(ctypes.Structure):
    _fields_ = [("n", ctypes.c_uint64), ("mismatches", ctypes.c_uint64),
                ("first_mismatch", ctypes.c_int64),
                ("max_abs_err", ctypes.c_double), ("max_rel_err", ctypes.c_double),
                ("err_sum", ctypes.c_double),
                ("nan_ref", ctypes.c_uint64), ("nan_cand", ctypes.c_uint64),
                ("inf_ref", ctypes.c_uint64), ("inf_cand", ctypes.c_uint64)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class Segment(ctypes.Structure):
    _fields_ = [("ref", ctypes.c_void_p), ("cand", ctypes.c_void_p),
                ("n", ctypes.c_uint64), ("dtype", ctypes.c_int32),
                ("rtol", ctypes.c_double), ("atol", ctypes.c_double),
                ("equal_nan", ctypes.c_int32)]


_lib = None


def lib():
    """Load the compiled oracle, building it first if it is not there."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _b
            _b.build()
        L = ctypes.CDLL(LIB_PATH)
        u32p = ctypes.POINTER(ctypes.c_uint32)
        L.or_philox4x32_10.argtypes = [u32p, u32p, u32p]
        L.or_philox_block.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64, u32p]
        L.or_ln_f32.argtypes = [ctypes.c_float]
        L.or_ln_f32.restype = ctypes.c_float
        L.or_sincos_2pi_f32.argtypes = [ctypes.c_uint32, ctypes.POINTER(ctypes.c_float),
                                        ctypes.POINTER(ctypes.c_float)]
        L.or_box_muller_f32.argtypes = [ctypes.c_uint32, ctypes.c_uint32,
                                        ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_float)]
        L.or_bf16_rne.argtypes = [ctypes.c_uint32]
        L.or_bf16_rne.restype = ctypes.c_uint16
        L.or_next_f32.argtypes = [ctypes.c_uint32, ctypes.c_int]
        L.or_next_f32.restype = ctypes.c_uint32
        L.or_next_bf16.argtypes = [ctypes.c_uint16, ctypes.c_int]
        L.or_next_bf16.restype = ctypes.c_uint16
        vp = ctypes.c_void_p
        L.or_philox_blocks.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                       ctypes.c_uint64, vp]
        L.or_ln_f32_n.argtypes = [vp, vp, ctypes.c_uint64]
        L.or_sincos_2pi_f32_n.argtypes = [vp, vp, vp, ctypes.c_uint64]
        L.or_sincos_table.argtypes = [vp, vp]
        L.or_bf16_rne_n.argtypes = [vp, vp, ctypes.c_uint64]
        L.or_f16_rne_n.argtypes = [vp, vp, ctypes.c_uint64]
        L.or_radius_f32_n.argtypes = [vp, vp, ctypes.c_uint64]
        L.or_performance.argtypes = [ctypes.c_double]
        L.or_performance.restype = ctypes.c_double
        L.or_reward.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_double]
        L.or_reward.restype = ctypes.c_double
        L.or_synth.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32,
                               ctypes.POINTER(DistParams), ctypes.c_uint64, ctypes.c_uint64,
                               ctypes.c_void_p]
        L.or_synth_at.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32,
                                  ctypes.POINTER(DistParams), ctypes.c_void_p, ctypes.c_uint64,
                                  ctypes.c_void_p]
        L.or_special_class_counts.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.POINTER(DistParams),
                                              ctypes.c_uint64, ctypes.c_uint64, vp]
        L.or_special_class_counts.restype = ctypes.c_int
        L.or_perturb.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int32,
                                 ctypes.POINTER(PerturbPlan), ctypes.c_uint64, ctypes.c_uint64,
                                 ctypes.c_void_p, ctypes.c_void_p]
        L.or_compare.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32,
                                 ctypes.c_double, ctypes.c_double, ctypes.c_int32,
                                 ctypes.POINTER(Report)]
        L.or_compare_batched.argtypes = [ctypes.POINTER(Segment), ctypes.c_uint32,
                                         ctypes.POINTER(Report)]
        for name in ("or_synth", "or_synth_at", "or_perturb", "or_compare", "or_compare_batched"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


def _check(rc, what):
    if rc != 0:
        raise OracleError("%s failed with code %d" % (what, rc))


def dist_params(**kw) -> DistParams:
    p = DistParams()
    for k, v in kw.items():
        setattr(p, k, v)
    return p


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


# ---------------------------------------------------------------- philox
def philox4x32_10(ctr, key):
    c = (ctypes.c_uint32 * 4)(*[int(x) & 0xFFFFFFFF for x in ctr])
    k = (ctypes.c_uint32 * 2)(*[int(x) & 0xFFFFFFFF for x in key])
    o = (ctypes.c_uint32 * 4)()
    lib().or_philox4x32_10(c, k, o)
    return list(o)


def philox_block(seed, stream, c):
    o = (ctypes.c_uint32 * 4)()
    lib().or_philox_block(seed, stream, c, o)
    return list(o)


def philox_blocks(seed, stream, c0, n) -> np.ndarray:
    """Blocks c0 .. c0+n-1 as an (n, 4) uint32 array."""
    out = np.empty((n, 4), dtype=np.uint32)
    lib().or_philox_blocks(seed, stream, c0, n, _ptr(out))
    return out


# ---------------------------------------------------------------- building blocks
def ln_f32_n(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    y = np.empty_like(x)
    lib().or_ln_f32_n(_ptr(x), _ptr(y), x.size)
    return y


def sincos_2pi_f32_n(j24):
    j = np.ascontiguousarray(j24, dtype=np.uint32)
    s = np.empty(j.size, np.float32)
    c = np.empty(j.size, np.float32)
    lib().or_sincos_2pi_f32_n(_ptr(j), _ptr(s), _ptr(c), j.size)
    return s, c


def radius_f32_n(k24) -> np.ndarray:
    """Box-Muller radius sqrt(-2 ln u1), u1 = (k24 + 1) 2^-24."""
    k = np.ascontiguousarray(k24, dtype=np.uint32)
    r = np.empty(k.size, np.float32)
    lib().or_radius_f32_n(_ptr(k), _ptr(r), k.size)
    return r


def bf16_rne_n(bits) -> np.ndarray:
    x = np.ascontiguousarray(bits, dtype=np.uint32)
    y = np.empty(x.size, np.uint16)
    lib().or_bf16_rne_n(_ptr(x), _ptr(y), x.size)
    return y


def f16_rne_n(bits) -> np.ndarray:
    """fp32 bit patterns -> IEEE binary16 bit patterns (round to nearest even)."""
    x = np.ascontiguousarray(bits, dtype=np.uint32)
    y = np.empty(x.size, np.uint16)
    lib().or_f16_rne_n(_ptr(x), _ptr(y), x.size)
    return y


def ln_f32(x: float) -> np.float32:
    return np.float32(lib().or_ln_f32(float(np.float32(x))))


def sincos_table():
    """The 256 table values (sin, cos of 2 pi k / 256 in fp32) of sincos_2pi_f32."""
    s = np.empty(256, np.float32)
    c = np.empty(256, np.float32)
    lib().or_sincos_table(_ptr(s), _ptr(c))
    return s, c


def sincos_2pi_f32(j24: int):
    s, c = ctypes.c_float(), ctypes.c_float()
    lib().or_sincos_2pi_f32(j24, ctypes.byref(s), ctypes.byref(c))
    return np.float32(s.value), np.float32(c.value)


def box_muller_f32(wa: int, wb: int):
    zc, zs = ctypes.c_float(), ctypes.c_float()
    lib().or_box_muller_f32(wa, wb, ctypes.byref(zc), ctypes.byref(zs))
    return np.float32(zc.value), np.float32(zs.value)


def bf16_rne(bits: int) -> int:
    return int(lib().or_bf16_rne(bits))


def next_f32(bits: int, up: bool) -> int:
    return int(lib().or_next_f32(bits, int(up)))


def next_bf16(bits: int, up: bool) -> int:
    return int(lib().or_next_bf16(bits, int(up)))


# ---------------------------------------------------------------- synthesis
def synth(seed, stream, dtype, dist, params: DistParams, n, offset=0) -> np.ndarray:
    """Elements [offset, offset+n) as raw storage (uint32 or uint16)."""
    out = np.empty(n, dtype=NP_STORAGE[dtype])
    _check(lib().or_synth(seed, stream, DTYPES[dtype], DISTS[dist], ctypes.byref(params),
                          offset, n, _ptr(out)), "or_synth")
    return out


def synth_at(seed, stream, dtype, dist, params: DistParams, idx) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.uint64)
    out = np.empty(idx.size, dtype=NP_STORAGE[dtype])
    _check(lib().or_synth_at(seed, stream, DTYPES[dtype], DISTS[dist], ctypes.byref(params),
                             _ptr(idx), idx.size, _ptr(out)), "or_synth_at")
    return out


def special_class_counts(seed, stream, params: DistParams, n, offset=0) -> np.ndarray:
    """[NaN, Inf, denormal, zero, normal] counts of SPECIAL elements [offset, offset+n)."""
    out = np.zeros(5, dtype=np.uint64)
    _check(lib().or_special_class_counts(seed, stream, ctypes.byref(params), offset, n, _ptr(out)),
           "or_special_class_counts")
    return out


# ---------------------------------------------------------------- candidates
def perturb(seed, stream, dtype, op, ref: np.ndarray, cand: np.ndarray = None, *, p=0.0,
            value=0.0, bits=0, idx=None, offset=0) -> np.ndarray:
    """Apply one derivation step to the window [offset, offset+len(ref)).

    Elementwise ops write every element of cand from ref; index ops write only
    listed elements (cand defaults to a copy of ref)."""
    ref = np.ascontiguousarray(ref)
    if cand is None:
        cand = ref.copy()
    idx_arr = np.ascontiguousarray(idx if idx is not None else [], dtype=np.uint64)
    plan = PerturbPlan()
    plan.op = OPS[op]
    plan.p = p
    plan.value = value
    plan.bits = bits & 0xFFFFFFFF
    plan.idx = idx_arr.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64))
    plan.nidx = idx_arr.size
    _check(lib().or_perturb(seed, stream, DTYPES[dtype], ctypes.byref(plan), offset, ref.size,
                            _ptr(ref), _ptr(cand)), "or_perturb")
    return cand


# ---------------------------------------------------------------- Eq. (1)
def compare(ref: np.ndarray, cand: np.ndarray, dtype, rtol, atol, equal_nan) -> dict:
    ref = np.ascontiguousarray(ref)
    cand = np.ascontiguousarray(cand)
    assert ref.size == cand.size
    r = Report()
    _check(lib().or_compare(_ptr(ref), _ptr(cand), ref.size, DTYPES[dtype], rtol, atol,
                            int(bool(equal_nan)), ctypes.byref(r)), "or_compare")
    return r.as_dict()


def compare_batched(segments) -> list:
    """segments: list of (ref, cand, dtype, rtol, atol, equal_nan)."""
    keep = []
    arr = (Segment * max(1, len(segments)))()
    for k, (ref, cand, dtype, rtol, atol, eqn) in enumerate(segments):
        ref = np.ascontiguousarray(ref)
        cand = np.ascontiguousarray(cand)
        keep += [ref, cand]
        arr[k] = Segment(ref.ctypes.data, cand.ctypes.data, ref.size, DTYPES[dtype], rtol, atol,
                         int(bool(eqn)))
    reps = (Report * max(1, len(segments)))()
    _check(lib().or_compare_batched(arr, len(segments), reps), "or_compare_batched")
    return [reps[k].as_dict() for k in range(len(segments))]


# ---------------------------------------------------------------- Eq. (3), Eq. (4)
def performance(mean_latency_ms: float) -> float:
    """Eq. (3): P = 1 / latency (latency in ms, P in 1/ms)."""
    return lib().or_performance(mean_latency_ms)


def reward(compiled: int, valid: int, p: float) -> float:
    """Eq. (4): r = -1 + C + C V P."""
    return lib().or_reward(int(compiled), int(valid), float(p))

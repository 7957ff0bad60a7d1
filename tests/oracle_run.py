"""Run a workload case through the CPU oracle (test helper).

Builds the reference tensor and the candidate exactly as the case describes,
using only the oracle; the GPU tests call this to get expected values.
"""
import numpy as np

import oracle as O


def params_of(spec):
    return O.dist_params(**spec.params)


def oracle_ref(spec, offset=0, n=None):
    n = spec.n - offset if n is None else n
    return O.synth(spec.seed, spec.stream, spec.dtype, spec.dist, params_of(spec), n, offset=offset)


def oracle_cand(case, ref, offset=0):
    """Apply the case's derivation steps to the window [offset, offset+len(ref))."""
    cand = ref.copy()
    for s in case.steps:
        if s.op in ("copy", "ulp", "scale", "special_flip"):
            cand = O.perturb(s.seed, s.stream, case.ref.dtype, s.op, ref, np.empty_like(ref),
                             p=s.p, value=s.value, offset=offset)
        else:
            cand = O.perturb(s.seed, s.stream, case.ref.dtype, s.op, ref, cand, value=s.value,
                             bits=s.bits, idx=s.idx, offset=offset)
    return cand


def oracle_case(case):
    ref = oracle_ref(case.ref)
    cand = oracle_cand(case, ref)
    rep = O.compare(ref, cand, case.ref.dtype, case.rtol, case.atol, case.equal_nan)
    return ref, cand, rep


def oracle_elements(case, idx):
    """Reference and candidate values at global indices idx, one element at a time."""
    idx = np.asarray(idx, dtype=np.uint64)
    ref = O.synth_at(case.ref.seed, case.ref.stream, case.ref.dtype, case.ref.dist,
                     params_of(case.ref), idx)
    cand = np.empty_like(ref)
    for k, i in enumerate(idx):
        cand[k] = oracle_cand(case, ref[k:k + 1], offset=int(i))[0]
    return ref, cand


# ------------------------------------------------------------ chunked runs
# The oracle is serial; these helpers only split a large tensor into windows
# and run the serial oracle on each window from a thread pool (ctypes releases
# the GIL), to keep full-size parity tests within seconds.
import os
from concurrent.futures import ThreadPoolExecutor


def workers():
    return max(1, min(16, os.cpu_count() or 1))


def _windows(n, parts):
    step = max(1, -(-n // parts))
    return [(o, min(step, n - o)) for o in range(0, n, step)]


def windowed(n, size):
    """(offset, length) of consecutive windows of at most `size` elements."""
    return [(o, min(size, n - o)) for o in range(0, n, size)]


def oracle_ref_parallel(spec, offset=0, n=None):
    """Elements [offset, offset + n) of the reference (default: all of it)."""
    n = spec.n - offset if n is None else n
    out = np.empty(n, dtype=O.NP_STORAGE[spec.dtype])
    def run(w):
        o, m = w
        out[o:o + m] = oracle_ref(spec, offset + o, m)
    with ThreadPoolExecutor(workers()) as ex:
        list(ex.map(run, _windows(n, 4 * workers())))
    return out


def oracle_cand_parallel(case, ref, offset=0):
    """The candidate over the window of `ref`, which starts at element `offset`."""
    cand = np.empty_like(ref)
    def run(w):
        o, m = w
        cand[o:o + m] = oracle_cand(case, ref[o:o + m], offset=offset + o)
    with ThreadPoolExecutor(workers()) as ex:
        list(ex.map(run, _windows(ref.size, 4 * workers())))
    return cand


def oracle_case_parallel(case):
    ref = oracle_ref_parallel(case.ref)
    cand = oracle_cand_parallel(case, ref)
    rep = O.compare(ref, cand, case.ref.dtype, case.rtol, case.atol, case.equal_nan)
    return ref, cand, rep


def special_counts_parallel(spec):
    p = params_of(spec)
    with ThreadPoolExecutor(workers()) as ex:
        parts = list(ex.map(lambda w: O.special_class_counts(spec.seed, spec.stream, p, w[1], offset=w[0]),
                            _windows(spec.n, 4 * workers())))
    return np.sum(parts, axis=0)

"""Throughput of the synthesis + check path on one MI355X.

A step is one pass of the whole path over one batch of synthetic input:
synthesize the reference tensor(s) (sv_synth; sv_synth_batched for the
batched workloads), check the candidates against them under Eq. (1)
(sv_compare; sv_compare_batched), and bring the report(s) to the host.  Candidates are derived
once before timing (workload support, untimed).  Inputs are resident in HBM
when the timed region starts.  Steps are pipelined by one: step k's synthesis
and check are queued (sv_compare_submit) before the host waits for step k-1's
reports (sv_compare_wait), so the GPU does not idle while a report travels to
the host; every report of the K steps is on the host before the clock stops.
sync_ms_per_step times the same steps with each one waited for before the
next is queued.  The W warm-up steps are followed by more untimed steps until
the warm-up has lasted 100 ms (the GPU raises its clocks under load).

value = (bytes synthesized + bytes checked) / time per step, in GB/s
(1e9 bytes/s): synthesis writes n * itemsize bytes, the check reads
2 * n * itemsize bytes (algorithmic bytes); with an early-exit check
(candidates_round) a failing segment counts only the bytes up to and
including its first mismatch.

The default workload is the 2^30-element fp32 special-value stream (4 GiB
reference, 12 GiB of algorithmic traffic per step).  After the timed passes a
cold pass repeats the steps with a 1 GiB write before each one (evicting the
256 MB Infinity Cache and the L2) and reports the kernels' durations there
(`cold`): the warm figures of workloads that fit the cache are not HBM
figures.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                       [--no-cpu-baseline] [--copy-probe] [--perf-stage]
"""
import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E, AMD public figure
ELEMENTWISE = ("copy", "ulp", "scale", "special_flip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
# the workloads of workloads.py (listed here so that a wrong name fails before the GPU is touched)
WORKLOAD_NAMES = ("uniform_small", "normal_ulp", "bf16_batch", "ragged_batch", "special_stream", "candidates_round")
EVICT_BYTES = 1 << 30     # written before each step of the cold pass


def kernel_source_hash():
    """Hash of the library sources (comments and blank lines removed) and build
    flags: the HBM-traffic counters in profiles/ are reported only while the
    code they were taken on is unchanged."""
    import hashlib
    import re
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_00058_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name)) as f:
            code = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
        code = "\n".join(l for l in (re.sub(r"//.*", "", x).rstrip() for x in code.split("\n")) if l)
        h.update(name.encode() + code.encode())
    with open(os.path.join(ROOT, "paper_2609_00058_amd", "build.py"), "rb") as f:
        h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, role):
    """HBM bytes per launch of the workload's synthesis or check kernel (role
    "synth" / "compare") from the committed rocprofv3 counter summary, or None
    when the counters were taken on other sources or not on this workload."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_hash") != kernel_source_hash():
        return None
    k = t.get("workloads", {}).get(workload, {}).get(role)
    return k["hbm_bytes"] if k else None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="special_stream", choices=WORKLOAD_NAMES)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--full-check", action="store_true",
                    help="check failing segments in full even where the workload stops at the first mismatch")
    ap.add_argument("--files", action="store_true",
                    help="time synthesis into a file and the check of two files instead (1 GiB fp32 each)")
    ap.add_argument("--perf-stage", action="store_true",
                    help="time the fail-fast sequence on a synthetic candidate kernel instead (Eq. 3-4)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="copy 256 MiB device-to-device once before timing (known-size kernel for "
                         "calibrating the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.steps < 1 or args.warmup < 0:
        ap.error("--steps must be at least 1 and --warmup at least 0")
    return args


def stream_copy_GBps(torch):
    """A STREAM-like reference on the same GPU: a 512 MiB device-to-device copy
    (torch's copy kernel), bytes read + written per second, best of 20."""
    src = torch.ones(1 << 27, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    best = None
    for _ in range(23):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        dst.copy_(src)
        b.record()
        b.synchronize()
        ms = a.elapsed_time(b)
        best = ms if best is None or ms < best else best
    del src, dst
    return round(2 * (1 << 29) / (best * 1e-3) / 1e9, 1)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def host_threads():
    """Threads for the all-core leg: the CPUs this process may run on, at most
    16 (the host share of one GPU)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def merge_reports(parts):
    """Reports of consecutive windows of one tensor, (offset, report) in order,
    merged into the tensor's: counts add, the first index is the earliest
    window's, maxima take the maximum, the fp64 sums are added in window order
    with Neumaier's compensation."""
    out = dict(parts[0][1])
    out["first_mismatch"] = -1
    out["n"] = out["mismatches"] = out["nan_ref"] = out["nan_cand"] = out["inf_ref"] = out["inf_cand"] = 0
    out["max_abs_err"] = out["max_rel_err"] = 0.0
    s = c = 0.0
    for off, r in parts:
        if out["first_mismatch"] < 0 and r["first_mismatch"] >= 0:
            out["first_mismatch"] = off + r["first_mismatch"]
        for k in ("n", "mismatches", "nan_ref", "nan_cand", "inf_ref", "inf_cand"):
            out[k] += r[k]
        out["max_abs_err"] = max(out["max_abs_err"], r["max_abs_err"])
        out["max_rel_err"] = max(out["max_rel_err"], r["max_rel_err"])
        d = r["err_sum"]
        t = s + d
        c += ((s - t) + d) if abs(s) >= abs(d) else ((d - t) + s)
        s = t
    out["err_sum"] = s + c
    return out


def cpu_baseline(wl, min_seconds=6.0, max_elems=1 << 24):
    """The oracle, as it stands (serial C), timed on a bounded sample of one
    step of the workload: synthesis + check of the first max_elems elements of
    each of the first two tensors (a prefix synthesizes the same bits as the
    tensor's; the candidate is derived untimed, index faults past the prefix
    dropped).  Two legs, each repeated until min_seconds have been timed (at
    most 1000 times): one thread, and all host threads (up to 16), each
    thread running the serial oracle on its own window of every tensor, the
    windows' reports merged in order.  `value` is the all-threads leg."""
    import numpy as np
    from concurrent.futures import ThreadPoolExecutor
    import oracle as O
    cases = wl.cases if not wl.batched else wl.cases[:2]
    work = []
    for case in cases:
        spec = case.ref
        n = min(spec.n, max_elems)
        p = O.dist_params(**spec.params)
        ref = O.synth(spec.seed, spec.stream, spec.dtype, spec.dist, p, n)
        cand = ref.copy()
        for st in case.steps:
            if st.op in ELEMENTWISE:
                cand = O.perturb(st.seed, st.stream, spec.dtype, st.op, ref, np.empty_like(ref), p=st.p,
                                 value=st.value)
            else:
                idx = np.asarray(st.idx, dtype=np.uint64)
                cand = O.perturb(st.seed, st.stream, spec.dtype, st.op, ref, cand, value=st.value, bits=st.bits,
                                 idx=idx[idx < n])
        work.append((case, spec, p, n, cand))
    elems = sum(w[3] for w in work)
    nbytes_rep = sum(3 * w[3] * w[1].itemsize for w in work)

    def one_thread():
        for case, spec, p, n, cand in work:
            ref = O.synth(spec.seed, spec.stream, spec.dtype, spec.dist, p, n)
            O.compare(ref, cand, spec.dtype, case.rtol, case.atol, case.equal_nan)

    threads = host_threads()
    pool = ThreadPoolExecutor(threads)

    def all_threads():
        for case, spec, p, n, cand in work:
            step = -(-n // threads)
            wins = [(o, min(step, n - o)) for o in range(0, n, step)]

            def run(w):
                o, m = w
                ref = O.synth(spec.seed, spec.stream, spec.dtype, spec.dist, p, m, offset=o)
                return o, O.compare(ref, cand[o:o + m], spec.dtype, case.rtol, case.atol, case.equal_nan)
            merge_reports(list(pool.map(run, wins)))

    def timed(fn):
        secs, reps = 0.0, 0
        while reps < 1000 and (reps == 0 or secs < min_seconds):
            t0 = time.perf_counter()
            fn()
            secs += time.perf_counter() - t0
            reps += 1
        return reps, secs

    r1, s1 = timed(one_thread)
    rn, sn = timed(all_threads)
    pool.shutdown()
    return {"value": round(rn * nbytes_rep / sn / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": "synthesis + check of the first %d elements of %d tensor(s) (%d bytes of algorithmic "
                      "traffic), %d times on %d threads (each on its window) in %.1f s; %d times on one thread "
                      "in %.1f s" % (max_elems, len(work), nbytes_rep, rn, threads, sn, r1, s1),
            "value_1_thread": round(r1 * nbytes_rep / s1 / 1e9, 4),
            "cpu": cpu_model(), "host_cpus": os.cpu_count()}


def perf_stage(args):
    """The stages after the functional check (Eq. 3-4) on a synthetic candidate:
    z = a x + y over 2^26 fp32 elements (768 MiB of traffic per run), loaded
    from the test candidates' code object.  Functional check against a
    reference computed by torch, then the performance stage warm (back-to-back
    runs) and cold (Infinity Cache and L2 evicted before each run), then the
    reward.  `value` is P = 1 / mean latency of the warm runs."""
    import struct
    import torch
    import paper_2609_00058_amd as sv
    torch.cuda.set_device(0)
    with open(os.path.join(ROOT, "tests", "kernels", "candidates.hsaco"), "rb") as f:
        code = f.read()
    n = 1 << 26
    g = torch.Generator().manual_seed(0)
    x = torch.randn(n, generator=g).cuda()
    y = torch.randn(n, generator=g).cuda()
    z = torch.empty_like(x)
    a = 1.7
    ref = torch.tensor(a, device="cuda") * x + y
    argbuf = struct.pack("<QQQfxxxxQ", z.data_ptr(), x.data_ptr(), y.data_ptr(), a, n)
    grid, block = ((n + 255) // 256,), (256,)
    k = sv.kernel_load(code, "sv_test_axpy")
    k.launch(grid, block, argbuf)
    rep = sv.compare(ref, z, 0.0, 0.0)
    valid = rep["mismatches"] == 0
    warm = k.time(grid, block, argbuf, warmup=args.warmup, reps=args.steps)
    cold = k.time(grid, block, argbuf, warmup=1, reps=args.steps, flush_bytes=512 << 20)
    nbytes = 3 * 4 * n
    out = {"metric": "performance stage: P = 1 / mean latency of a candidate kernel (Eq. 3)",
           "value": round(warm["perf"], 4), "unit": "1/ms", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(warm["mean_ms"], 5), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
           "config": {"workload": "axpy_f32_67108864", "candidate": "sv_test_axpy", "bytes_per_run": nbytes},
           "functional_check": {"mismatches": rep["mismatches"], "valid": valid},
           "timing_warm": {k_: round(v, 6) for k_, v in warm.items()},
           "timing_cold": {k_: round(v, 6) for k_, v in cold.items()},
           "candidate_GBps_warm": round(nbytes / (warm["mean_ms"] * 1e-3) / 1e9, 1),
           "candidate_GBps_cold": round(nbytes / (cold["mean_ms"] * 1e-3) / 1e9, 1),
           "reward": sv.reward(True, valid, warm["perf"])}
    k.free()
    print(json.dumps(out), flush=True)


def files_stage(args):
    """Test data as files: sv_synth_file writes 2^28 fp32 normal(5, 10) values
    (1 GiB) to a file; sv_compare_file checks that file against a candidate
    file (the reference with +-1 ulp on 0.1 % of elements, written untimed).
    Each is timed over `steps` runs after one untimed run (synthesis into a
    new file each time), next to the rates of a plain 1 GiB write into a new
    file and a single-threaded 2 GiB read of the same files (page cache warm),
    which bound them.  `value` is the file check's GB/s."""
    import shutil
    import tempfile
    import numpy as np
    import torch
    import paper_2609_00058_amd as sv
    torch.cuda.set_device(0)
    n = 1 << 28
    d = tempfile.mkdtemp(prefix="sv_bench_", dir=os.environ.get("SV_BENCH_DIR", "/tmp"))
    try:
        rp, cp = os.path.join(d, "ref.bin"), os.path.join(d, "cand.bin")
        prm = dict(mean=5.0, std=10.0)
        sv.synth_file(rp, n, 0, 0, "f32", "normal", **prm)
        ref = torch.empty(n, device="cuda")
        sv.synth(ref, 0, 0, "normal", **prm)
        cand = torch.empty_like(ref)
        sv.perturb(ref, cand, 0, 1, "ulp", p=1e-3)
        cand.cpu().numpy().tofile(cp)
        del ref, cand
        torch.cuda.empty_cache()
        t = []
        for k in range(args.steps):
            sp = os.path.join(d, "synth%d.bin" % k)   # a new file: overwriting one first frees its cached pages
            t0 = time.perf_counter()
            sv.synth_file(sp, n, 0, 0, "f32", "normal", **prm)
            t.append(time.perf_counter() - t0)
            os.unlink(sp)
        synth_s = sorted(t)[len(t) // 2]
        sv.compare_file(rp, cp, n, "f32", 1e-6, 0.0)
        t = []
        for _ in range(args.steps):
            t0 = time.perf_counter()
            rep = sv.compare_file(rp, cp, n, "f32", 1e-6, 0.0)
            t.append(time.perf_counter() - t0)
        cmp_s = sorted(t)[len(t) // 2]
        buf = np.fromfile(rp, dtype=np.uint8)
        t0 = time.perf_counter()
        with open(os.path.join(d, "plain.bin"), "wb") as f:
            f.write(memoryview(buf))
        write_s = time.perf_counter() - t0
        t0 = time.perf_counter()
        for path in (rp, cp):
            with open(path, "rb") as f:
                while f.readinto(memoryview(buf)[: 64 << 20]):
                    pass
        read_s = time.perf_counter() - t0
        st = os.statvfs(d)
        nbytes = 4 * n
        out = {"metric": "file check throughput (GB/s of file bytes read)", "value": round(2 * nbytes / cmp_s / 1e9, 2),
               "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": 1, "ms_per_step": round(cmp_s * 1e3, 2),
               "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
               "data": "synthetic", "config": {"workload": "files_f32_268435456", "dir": d,
                                               "dir_free_GB": round(st.f_bavail * st.f_frsize / 1e9, 1)},
               "synth_file_GBps": round(nbytes / synth_s / 1e9, 2),
               "compare_file_GBps": round(2 * nbytes / cmp_s / 1e9, 2),
               "plain_write_GBps": round(nbytes / write_s / 1e9, 2),
               "plain_read_GBps": round(2 * nbytes / read_s / 1e9, 2),
               "report": {k: rep[k] for k in ("mismatches", "first_mismatch", "max_rel_err")}}
        print(json.dumps(out), flush=True)
    finally:
        shutil.rmtree(d, ignore_errors=True)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: the library runs the path on a single MI355X and has no "
              "multi-GPU execution; rerun with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if args.perf_stage:
        return perf_stage(args)
    if args.files:
        return files_stage(args)
    import torch
    import paper_2609_00058_amd as sv
    import workloads as W

    torch.cuda.set_device(0)
    wl = W.WORKLOADS[args.workload]()
    if args.full_check:
        wl.stop_at_first = False
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "i32": torch.int32}
    uniq, which = wl.ref_groups()
    refs = []
    for spec in uniq:
        r = torch.empty(spec.n, dtype=tdt[spec.dtype], device="cuda")
        sv.synth(r, spec.seed, spec.stream, spec.dist, **spec.params)
        refs.append(r)
    cands = []
    for case, j in zip(wl.cases, which):
        r = refs[j]
        c = torch.empty_like(r)
        for s in case.steps:
            if s.op in ELEMENTWISE:
                sv.perturb(r, c, s.seed, s.stream, s.op, p=s.p, value=s.value)
            else:
                sv.perturb(r, c, s.seed, s.stream, s.op, value=s.value, bits=s.bits, idx=s.idx)
        cands.append(c)
    segs = [(refs[j], c, k.rtol, k.atol, k.equal_nan) for c, k, j in zip(cands, wl.cases, which)]
    if args.copy_probe:
        src = torch.ones(1 << 26, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    torch.cuda.synchronize()

    # batches are marshalled once: the same descriptors every step
    jobs = sv.SynthBatch([(r, spec.seed, spec.stream, spec.dist, spec.params) for spec, r in zip(uniq, refs)])
    batch = sv.SegmentBatch(segs)

    if not wl.batched:   # one tensor: both calls marshalled once as well
        c0 = wl.cases[0]
        synth_call = sv.PreparedSynth(refs[0], c0.ref.seed, c0.ref.stream, c0.ref.dist, **c0.ref.params)
        check_call = sv.PreparedCheck(*segs[0])

    def submit():
        if wl.batched:
            sv.synth_batched(jobs)
            return sv.compare_batched_submit(batch, stop_at_first=wl.stop_at_first)
        synth_call()
        return check_call.submit()

    def reports(ticket):
        return ticket.wait(as_array=True)    # one record per segment, no Python object per report

    def step():
        return reports(submit())

    def pipelined(k):
        prev, last = None, None
        for _ in range(k):
            t = submit()
            if prev is not None:
                last = reports(prev)
            prev = t
        return reports(prev) if prev is not None else last

    pipelined(args.warmup)
    # the GPU raises its clocks over tens of milliseconds of load: after the W
    # warm-up steps, keep stepping (untimed) until 100 ms of warm-up have run
    t_w = time.perf_counter()
    while time.perf_counter() - t_w < 0.1:
        pipelined(20)
    # timed region: K steps, no event markers
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    reps = pipelined(args.steps)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    # the same K steps, each waited for before the next is queued
    torch.cuda.synchronize()
    ts0 = time.perf_counter()
    for _ in range(args.steps):
        sync_reps = step()
    torch.cuda.synchronize()
    ts1 = time.perf_counter()
    assert sync_reps.tobytes() == reps.tobytes()
    # the same K steps again with HIP events around every kernel (on the stream
    # the kernels run on), for the per-kernel durations
    kinds = ("synth", "compare", "finalize")
    sv.profile_enable(True)
    for k in kinds:
        sv.profile_read(k)
    t2 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    sv.profile_enable(False)
    kt = {k: sv.profile_read(k) for k in kinds}
    # cold: the same K steps, each after a 1 GiB write on the same stream (it
    # evicts the Infinity Cache and the L2), the kernels timed by the same events
    evict = torch.empty(EVICT_BYTES // 4, dtype=torch.int32, device="cuda")
    sv.profile_enable(True)
    for k in kinds:
        sv.profile_read(k)
    for i in range(args.steps):
        evict.fill_(i)
        step()
    torch.cuda.synchronize()
    sv.profile_enable(False)
    kc = {k: sv.profile_read(k) for k in kinds}
    del evict

    ms = (t1 - t0) / args.steps * 1e3
    sbytes, cbytes = wl.synth_bytes, wl.compare_bytes
    if wl.stop_at_first:
        # bytes a check must read to settle each verdict: a passing segment in full, a failing one
        # up to and including its first mismatch
        cbytes = sum(2 * (int(r["n"]) if r["mismatches"] == 0 else int(r["first_mismatch"]) + 1) * k.ref.itemsize
                     for r, k in zip(reps, wl.cases))
    value = (sbytes + cbytes) / (ms / 1e3) / 1e9
    kernels = {}
    for k, nbytes in (("synth", sbytes), ("compare", cbytes), ("finalize", 0)):
        cnt, tot = kt[k]
        kernels[k] = {"launches": cnt, "avg_ms": round(tot / max(cnt, 1), 6),
                      "ms_per_step": round(tot / args.steps, 6)}
        if nbytes:
            kernels[k]["GBps"] = round(nbytes / (tot / args.steps / 1e3) / 1e9, 1)
    kernels["profiled_ms_per_step"] = round((t3 - t2) / args.steps * 1e3, 4)
    # the two kernels alone: (bytes synthesized + bytes checked) / (synthesis time + check time)
    kt_ms = (kt["synth"][1] + kt["compare"][1]) / args.steps
    kernels["synth_and_check_GBps"] = round((sbytes + cbytes) / (kt_ms / 1e3) / 1e9, 1)
    kernels["synth_and_check_frac"] = round(kernels["synth_and_check_GBps"] / HBM_PEAK_GBS, 4)
    kernel_ms = sum(kt[k][1] for k in kinds) / args.steps
    kernels["tensors_per_s"] = round(len(wl.cases) / (kernel_ms / 1e3), 1)   # kernel time only
    cold = {"evict_bytes": EVICT_BYTES}
    for k, nbytes in (("synth", sbytes), ("compare", cbytes), ("finalize", 0)):
        cnt, tot = kc[k]
        cold[k + "_ms"] = round(tot / args.steps, 6)
        if nbytes:
            cold[k + "_GBps"] = round(nbytes / (tot / args.steps / 1e3) / 1e9, 1)
    kc_ms = (kc["synth"][1] + kc["compare"][1]) / args.steps
    cold["synth_and_check_GBps"] = round((sbytes + cbytes) / (kc_ms / 1e3) / 1e9, 1)
    cold["synth_and_check_frac"] = round(cold["synth_and_check_GBps"] / HBM_PEAK_GBS, 4)
    copy = stream_copy_GBps(torch)
    dom = max(("synth", "compare"), key=lambda k: kernels[k]["ms_per_step"])
    achieved = kernels[dom]["GBps"]
    out = {
        "metric": "synth+check throughput (GB/s of algorithmic HBM traffic) on 1 MI355X",
        "value": round(value, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4), "sync_ms_per_step": round((ts1 - ts0) / args.steps * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "+".join(sorted(set({"f32": "f32", "bf16": "bf16", "i32": "int32"}[c.ref.dtype]
                                     for c in wl.cases))),
        "data": "synthetic",
        "config": {"workload": wl.name, "description": wl.description, "tensors": len(wl.cases),
                   "elements": wl.total_elems, "synth_bytes": sbytes, "check_bytes": cbytes,
                   "frac_of_hbm_peak": round(value / HBM_PEAK_GBS, 4),
                   "stream_copy_GBps": copy, "tensors_per_s": round(len(wl.cases) / (ms / 1e3), 1),
                   "elements_per_s": round(wl.total_elems / (ms / 1e3), 1)},
        "kernels": kernels,
        "cold": cold,
        "roofline": {"kernel": dom, "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(wl.name, dom)},
        "mismatches": [int(r["mismatches"]) for r in reps][:8],
        "failing_segments": sum(1 for r in reps if r["mismatches"]),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

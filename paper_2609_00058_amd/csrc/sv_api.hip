// sv_api.hip -- the C ABI of libsynthverify (declared in include/sv.h):
// argument validation, per-device scratch, stream selection, kernel timing.
//
// Every entry point validates all of its arguments before it issues any HIP
// call, and reports failures as a status code plus a thread-local message.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "sv_internal.h"

using namespace sv;

namespace {

thread_local hipStream_t t_stream = nullptr;
thread_local std::string t_error;

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  t_error = buf;
  return code;
}

// The status and message carry the error to the caller, so the runtime's
// per-thread last error is cleared: a later hipGetLastError() of the caller
// (torch checks it after its own launches) must not see the library's failure.
int hip_fail(hipError_t e, const char *what) {
  (void)hipGetLastError();
  return fail(SV_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

#define SV_HIP(call, what)                      \
  do {                                          \
    hipError_t e_ = (call);                     \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

// ------------------------------------------------------------ per-device scratch
struct DeviceState {
  std::mutex mu;                 // serialises calls that use the scratch below
  int cus = 0;
  Partial *partials = nullptr;   // one per (workgroup, segment piece)
  size_t partials_cap = 0;
  SegDesc *table = nullptr;      // batched segment table
  size_t table_cap = 0;
  uint64_t *idx = nullptr;
  size_t idx_cap = 0;
  SegDesc *h_table = nullptr;    // pinned staging
  size_t h_table_cap = 0;
  sv_report *h_reports = nullptr;  // pinned, host-mapped, coherent: the kernel writes reports here
  sv_report *d_reports = nullptr;  // the device address of h_reports
  size_t h_reports_cap = 0;
  uint64_t *h_idx = nullptr;
  size_t h_idx_cap = 0;
  SynthJob *synth_table = nullptr;   // batched synthesis job table
  size_t synth_table_cap = 0;
  SynthJob *h_synth = nullptr;       // its pinned staging
  size_t h_synth_cap = 0;
  hipEvent_t synth_copied = nullptr; // staging -> table copy of the last batch done
  hipEvent_t synth_done = nullptr;   // last batch kernel done (table free to overwrite)
  bool synth_pending = false;        // the two events above have been recorded
  uint32_t *counters = nullptr;      // arrival counters of the check (zero between launches)
  size_t counters_cap = 0;
  uint64_t *h_done = nullptr;        // pinned, host-mapped, coherent: a check's last word written
  uint64_t *d_done = nullptr;        // its device address
  uint64_t seq = 0;                  // sequence number of the last check launched
};

std::mutex g_devices_mu;
std::vector<DeviceState *> g_devices;

int current_device(DeviceState **out) {
  int dev = 0;
  SV_HIP(hipGetDevice(&dev), "hipGetDevice");
  std::lock_guard<std::mutex> g(g_devices_mu);
  if ((size_t)dev >= g_devices.size()) g_devices.resize(dev + 1, nullptr);
  if (!g_devices[dev]) {
    int cus = 0;
    SV_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev),
           "hipDeviceGetAttribute(multiProcessorCount)");
    auto *s = new DeviceState;
    s->cus = cus > 0 ? cus : 1;
    g_devices[dev] = s;
  }
  *out = g_devices[dev];
  return SV_OK;
}

int cu_count(int *cus) {
  DeviceState *ds;
  int rc = current_device(&ds);
  if (rc) return rc;
  *cus = ds->cus;
  return SV_OK;
}

template <class T>
int ensure_device(T *&ptr, size_t &cap, size_t need, const char *what) {
  if (need <= cap) return SV_OK;
  const size_t want = std::max(need, cap + cap / 2);
  if (ptr) (void)hipFree(ptr);
  ptr = nullptr;
  cap = 0;
  hipError_t e = hipMalloc((void **)&ptr, want * sizeof(T));
  if (e != hipSuccess) {
    ptr = nullptr;
    return fail(SV_ERR_ALLOC, "hipMalloc of %zu bytes for %s: %s", want * sizeof(T), what, hipGetErrorString(e));
  }
  cap = want;
  return SV_OK;
}

int ensure_reports(DeviceState *ds, size_t need) {
  if (need <= ds->h_reports_cap) return SV_OK;
  const size_t want = std::max(need, ds->h_reports_cap + ds->h_reports_cap / 2);
  if (ds->h_reports) (void)hipHostFree(ds->h_reports);
  ds->h_reports = nullptr;
  ds->d_reports = nullptr;
  ds->h_reports_cap = 0;
  hipError_t e = hipHostMalloc((void **)&ds->h_reports, want * sizeof(sv_report),
                               hipHostMallocMapped | hipHostMallocCoherent);
  if (e != hipSuccess) {
    ds->h_reports = nullptr;
    return fail(SV_ERR_ALLOC, "hipHostMalloc of %zu bytes for reports: %s", want * sizeof(sv_report),
                hipGetErrorString(e));
  }
  e = hipHostGetDevicePointer((void **)&ds->d_reports, ds->h_reports, 0);
  if (e != hipSuccess) {
    (void)hipHostFree(ds->h_reports);
    ds->h_reports = nullptr;
    return hip_fail(e, "hipHostGetDevicePointer(reports)");
  }
  ds->h_reports_cap = want;
  return SV_OK;
}

int ensure_counters(DeviceState *ds, size_t need) {
  if (need <= ds->counters_cap) return SV_OK;
  int rc = ensure_device(ds->counters, ds->counters_cap, need, "arrival counters");
  if (rc) return rc;
  SV_HIP(hipMemset(ds->counters, 0, ds->counters_cap * sizeof(uint32_t)), "hipMemset(arrival counters)");
  return SV_OK;
}

int ensure_done(DeviceState *ds) {
  if (ds->h_done) return SV_OK;
  hipError_t e = hipHostMalloc((void **)&ds->h_done, 64, hipHostMallocMapped | hipHostMallocCoherent);
  if (e != hipSuccess) {
    ds->h_done = nullptr;
    return fail(SV_ERR_ALLOC, "hipHostMalloc of the completion word: %s", hipGetErrorString(e));
  }
  e = hipHostGetDevicePointer((void **)&ds->d_done, ds->h_done, 0);
  if (e != hipSuccess) {
    (void)hipHostFree(ds->h_done);
    ds->h_done = nullptr;
    return hip_fail(e, "hipHostGetDevicePointer(completion word)");
  }
  *(volatile uint64_t *)ds->h_done = ds->seq;
  return SV_OK;
}

// Waits until the check launched with sequence number `seq` has written its
// reports: spins on the host-mapped completion word (a few hundred ns after
// the kernel's last store, well before a stream synchronisation would
// return), asking the stream now and then whether it failed instead.
int wait_done(DeviceState *ds, uint64_t seq, hipStream_t st) {
  using clock = std::chrono::steady_clock;
  const volatile uint64_t *flag = ds->h_done;
  std::chrono::microseconds interval(50);
  auto next = clock::now() + interval;
  while (*flag != seq) {
    __builtin_ia32_pause();
    const auto now = clock::now();
    if (now < next) continue;
    const hipError_t e = hipStreamQuery(st);
    if (e == hipSuccess) {
      if (*flag == seq) break;
      return fail(SV_ERR_HIP, "the check kernel finished without writing its reports");
    }
    if (e != hipErrorNotReady) return hip_fail(e, "waiting for the check");
    interval = std::min(interval * 2, std::chrono::microseconds(1000));
    next = now + interval;
  }
  std::atomic_thread_fence(std::memory_order_acquire);
  return SV_OK;
}

template <class T>
int ensure_pinned(T *&ptr, size_t &cap, size_t need, const char *what) {
  if (need <= cap) return SV_OK;
  const size_t want = std::max(need, cap + cap / 2);
  if (ptr) (void)hipHostFree(ptr);
  ptr = nullptr;
  cap = 0;
  hipError_t e = hipHostMalloc((void **)&ptr, want * sizeof(T), hipHostMallocDefault);
  if (e != hipSuccess) {
    ptr = nullptr;
    return fail(SV_ERR_ALLOC, "hipHostMalloc of %zu bytes for %s: %s", want * sizeof(T), what,
                hipGetErrorString(e));
  }
  cap = want;
  return SV_OK;
}

// ------------------------------------------------------------ kernel timing
struct ProfRecord {
  int kind;
  hipEvent_t start, stop;
};
std::atomic<int> g_prof_on{0};
std::mutex g_prof_mu;
std::vector<ProfRecord> g_prof;
std::vector<hipEvent_t> g_event_pool;

hipEvent_t take_event() {
  std::lock_guard<std::mutex> g(g_prof_mu);
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void push_record(int kind, hipEvent_t a, hipEvent_t b) {
  if (!a || !b) return;
  std::lock_guard<std::mutex> g(g_prof_mu);
  g_prof.push_back({kind, a, b});
}

// ------------------------------------------------------------ validation helpers
bool valid_dtype(int32_t d) { return d >= SV_F32 && d <= SV_I64; }
bool int_dtype(int32_t d) { return d == SV_I32 || d == SV_U8 || d == SV_I64; }
size_t elem_size(int32_t d) { return item_bytes(d); }

// The candidate steps each element type supports.
bool op_supported(int32_t dtype, int32_t op) {
  if (op == SV_OP_COPY || op == SV_OP_FAULT_AT) return true;
  switch (dtype) {
    case SV_F32: case SV_BF16: return true;
    case SV_I32: case SV_U8: return op == SV_OP_SET_AT;
    case SV_F16: return op == SV_OP_ULP || op == SV_OP_SET_AT;
    case SV_F64: return op == SV_OP_ULP;
    default: return false;
  }
}
constexpr uint64_t kMaxElems = 1ull << 60;

int check_tensor(const void *p, uint64_t n, int32_t dtype, const char *name) {
  if (n > kMaxElems) return fail(SV_ERR_INVALID_ARG, "%s: n = %llu exceeds 2^60", name, (unsigned long long)n);
  if (n && !p) return fail(SV_ERR_INVALID_ARG, "%s is NULL with n = %llu", name, (unsigned long long)n);
  if (n && ((uintptr_t)p % elem_size(dtype)))
    return fail(SV_ERR_INVALID_ARG, "%s = %p is not aligned to its %zu-byte elements", name, p, elem_size(dtype));
  return SV_OK;
}

int check_tolerances(double rtol, double atol) {
  if (!(rtol >= 0.0) || !std::isfinite(rtol)) return fail(SV_ERR_INVALID_ARG, "rtol = %g must be finite and >= 0", rtol);
  if (!(atol >= 0.0) || !std::isfinite(atol)) return fail(SV_ERR_INVALID_ARG, "atol = %g must be finite and >= 0", atol);
  return SV_OK;
}

uint64_t width32(double p) { return (uint64_t)std::floor(p * 4294967296.0); }

int check_seg(const sv_segment &g, uint32_t k) {
  if (!valid_dtype(g.dtype)) return fail(SV_ERR_UNSUPPORTED, "segment %u: unknown dtype %d", k, g.dtype);
  int rc = check_tensor(g.ref, g.n, g.dtype, "segment ref");
  if (!rc) rc = check_tensor(g.cand, g.n, g.dtype, "segment cand");
  if (!rc && !int_dtype(g.dtype)) rc = check_tolerances(g.rtol, g.atol);
  if (rc) t_error = "segment " + std::to_string(k) + ": " + t_error;
  return rc;
}

SegDesc make_desc(const sv_segment &g, uint64_t unit_begin) {
  SegDesc d;
  d.ref = g.ref;
  d.cand = g.cand;
  d.n = g.n;
  d.unit_begin = unit_begin;
  d.rtol = int_dtype(g.dtype) ? 0.0 : g.rtol;
  d.atol = int_dtype(g.dtype) ? 0.0 : g.atol;
  d.dtype = g.dtype;
  d.equal_nan = g.equal_nan ? 1 : 0;
  d.vec_ok = (((uintptr_t)g.ref | (uintptr_t)g.cand) & 15u) == 0 ? 1 : 0;
  d.pad = 0;
  return d;
}

void zero_report(sv_report *r, uint64_t n) {
  std::memset(r, 0, sizeof *r);
  r->n = n;
  r->first_mismatch = -1;
}

// grid for a check over `units` 16-byte units: at most SV_CMP_BLOCKS_PER_CU
// workgroups per CU, each owning whole waves of units
void compare_grid(uint64_t units, int cus, bool batched, uint32_t *nblocks, uint64_t *chunk) {
  const uint64_t per_iter = (uint64_t)kBlock;
  const uint64_t per_cu = batched ? SV_CMP_BATCH_BLOCKS_PER_CU : SV_CMP_BLOCKS_PER_CU;
  uint64_t nb = std::min<uint64_t>((units + per_iter - 1) / per_iter, (uint64_t)cus * per_cu);
  if (nb == 0) nb = 1;
  uint64_t c = (units + nb - 1) / nb;
  c = (c + kWave - 1) / kWave * kWave;       // whole waves of units per workgroup
  *chunk = c;
  *nblocks = (uint32_t)((units + c - 1) / c);
}

// The check kernel (and, for a batch, its finalize kernel), which write the
// reports into host-mapped memory and then the launch's sequence number; the
// host waits for that number.  Segments with no elements get their (empty)
// report here.
int run_compare(DeviceState *ds, CompareArgs &args, uint32_t nblocks, const sv_segment *segs, uint32_t nseg,
                sv_report *out, bool stop_at_first = false) {
  hipStream_t st = t_stream;
  int rc = ensure_device(ds->partials, ds->partials_cap, (size_t)nblocks + nseg, "partials");
  if (!rc) rc = ensure_reports(ds, nseg);
  if (!rc) rc = ensure_counters(ds, 1);
  if (!rc) rc = ensure_done(ds);
  if (rc) return rc;
  args.stop_at_first = stop_at_first ? 1 : 0;
  args.partials = ds->partials;
  args.counter = ds->counters;
  args.reports = ds->d_reports;
  args.done = ds->d_done;
  args.seq = ds->seq + 1;
  hipEvent_t e0 = nullptr, e1 = nullptr, e2 = nullptr;
  if (g_prof_on.load()) {
    e0 = take_event();
    e1 = take_event();
    e2 = take_event();
    if (e0) (void)hipEventRecord(e0, st);
  }
  uint32_t mask = 0;
  for (uint32_t k = 0; k < nseg; ++k) {
    const sv_segment *g = segs ? &segs[k] : nullptr;
    const uint64_t n = g ? g->n : args.single.n;
    if (n) mask |= 1u << (g ? g->dtype : args.single.dtype);
  }
  hipError_t e = launch_compare(args, nblocks, mask, st, e0 ? e1 : nullptr);
  if (e != hipSuccess) return hip_fail(e, "check kernel launch");
  ds->seq = args.seq;
  if (e0 && e1 && e2) {
    (void)hipEventRecord(e2, st);
    push_record(SV_PROF_COMPARE, e0, e1);
    push_record(SV_PROF_FINALIZE, e1, e2);
  }
  rc = wait_done(ds, args.seq, st);
  if (rc) return rc;
  for (uint32_t k = 0; k < nseg; ++k) {
    const uint64_t n = segs ? segs[k].n : args.single.n;
    if (n)
      out[k] = ds->h_reports[k];
    else
      zero_report(&out[k], 0);
    if (stop_at_first && out[k].mismatches) {   // only the verdict and the first index are defined
      const int64_t first = out[k].first_mismatch;
      zero_report(&out[k], n);
      out[k].mismatches = 1;
      out[k].first_mismatch = first;
    }
  }
  return SV_OK;
}

// Validates the arguments of one synthesis and prepares its kernel
// parameters; issues no HIP call.
int prepare_synth(uint64_t seed, uint64_t stream_id, int32_t dtype, int32_t dist, const sv_dist_params *params,
                  uint64_t n, void *out, SynthParams *pp) {
  if (!valid_dtype(dtype)) return fail(SV_ERR_UNSUPPORTED, "sv_synth: unknown dtype %d", dtype);
  if (dist < SV_UNIFORM || dist > SV_SPECIAL) return fail(SV_ERR_UNSUPPORTED, "sv_synth: unknown dist %d", dist);
  if ((dist == SV_INT_RANGE) != int_dtype(dtype))
    return fail(SV_ERR_UNSUPPORTED, "sv_synth: dist %d cannot produce dtype %d", dist, dtype);
  if (!params) return fail(SV_ERR_INVALID_ARG, "sv_synth: params is NULL");
  int rc = check_tensor(out, n, dtype, "sv_synth out");
  if (rc) return rc;
  SynthParams &p = *pp;
  std::memset(&p, 0, sizeof p);
  p.k0 = (uint32_t)seed;
  p.k1 = (uint32_t)(seed >> 32);
  p.s0 = (uint32_t)stream_id;
  p.s1 = (uint32_t)(stream_id >> 32);
  if (dist == SV_UNIFORM && dtype == SV_F64) {
    const double a = params->a, b = params->b, span = b - a;
    if (!(a < b) || !std::isfinite(a) || !std::isfinite(b) || !std::isfinite(span))
      return fail(SV_ERR_INVALID_ARG, "sv_synth: uniform needs finite a < b with finite b - a (a=%g b=%g)",
                  params->a, params->b);
    p.a64 = a;
    p.span64 = span;
  } else if (dist == SV_UNIFORM) {
    const float a = (float)params->a, b = (float)params->b;
    const float span = b - a;
    if (!(a < b) || !std::isfinite(a) || !std::isfinite(b) || !std::isfinite(span))
      return fail(SV_ERR_INVALID_ARG, "sv_synth: uniform needs finite fp32 a < b with finite b - a (a=%g b=%g)",
                  params->a, params->b);
    p.a = a;
    p.span = span;
  } else if (dist == SV_NORMAL || dist == SV_SPECIAL) {
    p.mean = (float)params->mean;
    p.std = (float)params->std;
    if (!std::isfinite(p.mean) || !std::isfinite(p.std) || !(p.std >= 0.0f))
      return fail(SV_ERR_INVALID_ARG, "sv_synth: normal needs finite fp32 mean and std >= 0 (mean=%g std=%g)",
                  params->mean, params->std);
    if (dist == SV_SPECIAL) {
      const double ps[4] = {params->p_nan, params->p_inf, params->p_denorm, params->p_zero};
      double tot = 0.0;
      for (double q : ps) {
        if (!(q >= 0.0 && q <= 1.0)) return fail(SV_ERR_INVALID_ARG, "sv_synth: class probability %g not in [0,1]", q);
        tot += q;
      }
      if (!(tot <= 1.0)) return fail(SV_ERR_INVALID_ARG, "sv_synth: class probabilities sum to %g > 1", tot);
      p.t_nan = width32(params->p_nan);
      p.t_inf = p.t_nan + width32(params->p_inf);
      p.t_den = p.t_inf + width32(params->p_denorm);
      p.t_zero = p.t_den + width32(params->p_zero);
    }
  } else {
    const int64_t lo = params->lo, hi = params->hi;
    const bool inside = dtype == SV_I64 ? true
                        : dtype == SV_U8 ? (lo >= 0 && hi <= 255)
                                         : (lo >= INT32_MIN && hi <= INT32_MAX);
    if (lo > hi || !inside)
      return fail(SV_ERR_INVALID_ARG, "sv_synth: integer range [%lld, %lld] must be non-empty and within %s",
                  (long long)lo, (long long)hi, dtype == SV_U8 ? "uint8" : dtype == SV_I64 ? "int64" : "int32");
    p.lo = lo;
    p.range = (uint64_t)hi - (uint64_t)lo + 1u;   // 0 for the whole int64 range
  }
  return SV_OK;
}

}  // namespace

namespace sv {
hipStream_t api_stream() { return t_stream; }
void api_clear_error() { t_error.clear(); }
int api_fail(int code, const char *msg) { return fail(code, "%s", msg); }
int api_hip_fail(hipError_t e, const char *what) { return hip_fail(e, what); }
}  // namespace sv

// =================================================================== C ABI
extern "C" {

int sv_abi_version(void) { return SV_ABI_VERSION; }

const char *sv_last_error(void) { return t_error.c_str(); }

int sv_set_stream(void *hip_stream) {
  t_stream = (hipStream_t)hip_stream;
  return SV_OK;
}

int sv_synth(uint64_t seed, uint64_t stream_id, int32_t dtype, int32_t dist, const sv_dist_params *params,
             uint64_t n, void *out) {
  return sv_synth_window(seed, stream_id, dtype, dist, params, 0, n, out);
}

int sv_synth_window(uint64_t seed, uint64_t stream_id, int32_t dtype, int32_t dist, const sv_dist_params *params,
                    uint64_t offset, uint64_t n, void *out) {
  t_error.clear();
  SynthParams p;
  int rc = prepare_synth(seed, stream_id, dtype, dist, params, n, out, &p);
  if (rc) return rc;
  if (offset > kMaxElems || n > kMaxElems - offset)
    return fail(SV_ERR_INVALID_ARG, "sv_synth_window: offset + n exceeds 2^60");
  const uint64_t per_block =
      dist == SV_SPECIAL ? 1 : (dist == SV_INT_RANGE || (dist == SV_UNIFORM && dtype == SV_F64)) ? 2 : 4;
  p.e0 = offset;
  p.c0 = offset / per_block;
  if (!n) return SV_OK;
  int cus;
  rc = cu_count(&cus);
  if (rc) return rc;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (g_prof_on.load()) {
    e0 = take_event();
    e1 = take_event();
    if (e0) (void)hipEventRecord(e0, t_stream);
  }
  SV_HIP(launch_synth(dtype, dist, p, n, out, cus, t_stream), "synthesis kernel launch");
  if (e0 && e1) {
    (void)hipEventRecord(e1, t_stream);
    push_record(SV_PROF_SYNTH, e0, e1);
  }
  return SV_OK;
}

// Jobs of the fp32 / bf16 / int32 kinds share one launch through a job table;
// jobs of the other element types (fp16, fp64, uint8, int64) are launched one
// by one after it (keeping the batched kernel's register budget to the kinds
// the batched workloads use).
static bool table_kind(int32_t dtype) { return dtype == SV_F32 || dtype == SV_BF16 || dtype == SV_I32; }

int sv_synth_batched(const sv_synth_job *jobs, uint32_t njobs) {
  t_error.clear();
  if (njobs == 0) return SV_OK;
  if (!jobs) return fail(SV_ERR_INVALID_ARG, "sv_synth_batched: jobs is NULL");
  std::vector<SynthParams> params(njobs);
  std::vector<uint32_t> table_jobs, direct_jobs;
  uint64_t tiles = 0;
  for (uint32_t k = 0; k < njobs; ++k) {
    const sv_synth_job &j = jobs[k];
    int rc = prepare_synth(j.seed, j.stream_id, j.dtype, j.dist, &j.params, j.n, j.out, &params[k]);
    if (rc) {
      t_error = "job " + std::to_string(k) + ": " + t_error;
      return rc;
    }
    if (!j.n) continue;
    if (!table_kind(j.dtype)) {
      direct_jobs.push_back(k);
      continue;
    }
    table_jobs.push_back(k);
    tiles += (units_of(j.dtype, j.n) + kBlock - 1) / kBlock;
  }
  if (table_jobs.empty() && direct_jobs.empty()) return SV_OK;
  DeviceState *ds;
  int rc = current_device(&ds);
  if (rc) return rc;
  std::lock_guard<std::mutex> lock(ds->mu);
  hipStream_t st = t_stream;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (g_prof_on.load()) {
    e0 = take_event();
    e1 = take_event();
  }
  const uint32_t nt = (uint32_t)table_jobs.size();
  if (nt) {
    if (!ds->synth_copied) {
      SV_HIP(hipEventCreateWithFlags(&ds->synth_copied, hipEventDisableTiming), "hipEventCreate");
      SV_HIP(hipEventCreateWithFlags(&ds->synth_done, hipEventDisableTiming), "hipEventCreate");
    }
    if (ds->synth_pending) {
      // the staging buffer is rewritten below: its last copy must have left it;
      // the device table is rewritten on this stream after the last batch read it
      SV_HIP(hipEventSynchronize(ds->synth_copied), "wait for the previous job-table copy");
      SV_HIP(hipStreamWaitEvent(st, ds->synth_done, 0), "order after the previous batch");
    }
    rc = ensure_pinned(ds->h_synth, ds->h_synth_cap, nt, "job table staging");
    if (!rc) rc = ensure_device(ds->synth_table, ds->synth_table_cap, nt, "job table");
    if (rc) return rc;
    uint64_t begin = 0;
    for (uint32_t t = 0; t < nt; ++t) {
      const sv_synth_job &j = jobs[table_jobs[t]];
      SynthJob &d = ds->h_synth[t];
      d.p = params[table_jobs[t]];
      d.out = j.out;
      d.n = j.n;
      d.nvec = units_of(j.dtype, j.n);
      d.tile_begin = begin;
      d.kind = j.dist * 4 + j.dtype;
      d.vec_ok = ((uintptr_t)j.out & 15u) == 0 ? 1 : 0;
      begin += (d.nvec + kBlock - 1) / kBlock;
    }
    SV_HIP(hipMemcpyAsync(ds->synth_table, ds->h_synth, nt * sizeof(SynthJob), hipMemcpyHostToDevice, st),
           "job table copy to device");
    SV_HIP(hipEventRecord(ds->synth_copied, st), "hipEventRecord");
  }
  if (e0) (void)hipEventRecord(e0, st);
  if (nt) SV_HIP(launch_synth_batched(ds->synth_table, nt, tiles, ds->cus, st), "batched synthesis kernel launch");
  for (uint32_t k : direct_jobs)
    SV_HIP(launch_synth(jobs[k].dtype, jobs[k].dist, params[k], jobs[k].n, jobs[k].out, ds->cus, st),
           "synthesis kernel launch");
  if (e0 && e1) {
    (void)hipEventRecord(e1, st);
    push_record(SV_PROF_SYNTH, e0, e1);
  }
  if (nt) {
    SV_HIP(hipEventRecord(ds->synth_done, st), "hipEventRecord");
    ds->synth_pending = true;
  }
  return SV_OK;
}

int sv_compare(const void *ref, const void *cand, uint64_t n, int32_t dtype, double rtol, double atol,
               int32_t equal_nan, sv_report *report) {
  t_error.clear();
  if (!report) return fail(SV_ERR_INVALID_ARG, "sv_compare: report is NULL");
  const sv_segment g{ref, cand, n, dtype, rtol, atol, equal_nan};
  int rc = check_seg(g, 0);
  if (rc) return rc;
  if (!n) {
    zero_report(report, 0);
    return SV_OK;
  }
  DeviceState *ds;
  rc = current_device(&ds);
  if (rc) return rc;
  std::lock_guard<std::mutex> lock(ds->mu);
  CompareArgs args;
  std::memset(&args, 0, sizeof args);
  args.segs = nullptr;
  args.single = make_desc(g, 0);
  args.nseg = 1;
  args.total_units = units_of(dtype, n);
  uint32_t nblocks;
  compare_grid(args.total_units, ds->cus, false, &nblocks, &args.chunk);
  return run_compare(ds, args, nblocks, nullptr, 1, report);
}

int sv_compare_batched(const sv_segment *segs, uint32_t nseg, sv_report *reports) {
  return sv_compare_batched_mode(segs, nseg, SV_CHECK_FULL, reports);
}

int sv_compare_batched_mode(const sv_segment *segs, uint32_t nseg, int32_t mode, sv_report *reports) {
  t_error.clear();
  if (mode != SV_CHECK_FULL && mode != SV_CHECK_STOP_AT_FIRST)
    return fail(SV_ERR_UNSUPPORTED, "sv_compare_batched_mode: unknown mode %d", mode);
  if (nseg == 0) return SV_OK;
  if (!segs || !reports) return fail(SV_ERR_INVALID_ARG, "sv_compare_batched: segs or reports is NULL");
  uint64_t total = 0;
  for (uint32_t k = 0; k < nseg; ++k) {
    int rc = check_seg(segs[k], k);
    if (rc) return rc;
    total += units_of(segs[k].dtype, segs[k].n);
  }
  if (total == 0) {
    for (uint32_t k = 0; k < nseg; ++k) zero_report(&reports[k], 0);
    return SV_OK;
  }
  DeviceState *ds;
  int rc = current_device(&ds);
  if (rc) return rc;
  std::lock_guard<std::mutex> lock(ds->mu);
  rc = ensure_pinned(ds->h_table, ds->h_table_cap, nseg, "segment table staging");
  if (!rc) rc = ensure_device(ds->table, ds->table_cap, nseg, "segment table");
  if (rc) return rc;
  uint64_t begin = 0;
  for (uint32_t k = 0; k < nseg; ++k) {
    ds->h_table[k] = make_desc(segs[k], begin);
    begin += units_of(segs[k].dtype, segs[k].n);
  }
  SV_HIP(hipMemcpyAsync(ds->table, ds->h_table, nseg * sizeof(SegDesc), hipMemcpyHostToDevice, t_stream),
         "segment table copy to device");
  CompareArgs args;
  std::memset(&args, 0, sizeof args);
  args.segs = ds->table;
  args.nseg = nseg;
  args.total_units = total;
  uint32_t nblocks;
  compare_grid(total, ds->cus, true, &nblocks, &args.chunk);
  return run_compare(ds, args, nblocks, segs, nseg, reports, mode == SV_CHECK_STOP_AT_FIRST);
}

int sv_perturb(uint64_t seed, uint64_t stream_id, int32_t dtype, const sv_perturb_plan *plan, uint64_t n,
               const void *ref, void *cand) {
  t_error.clear();
  if (!plan) return fail(SV_ERR_INVALID_ARG, "sv_perturb: plan is NULL");
  if (!valid_dtype(dtype)) return fail(SV_ERR_UNSUPPORTED, "sv_perturb: unknown dtype %d", dtype);
  const int32_t op = plan->op;
  if (op < SV_OP_COPY || op > SV_OP_FAULT_AT) return fail(SV_ERR_UNSUPPORTED, "sv_perturb: unknown op %d", op);
  if (!op_supported(dtype, op))
    return fail(SV_ERR_UNSUPPORTED, "sv_perturb: op %d is not available for dtype %d", op, dtype);
  int rc = check_tensor(ref, n, dtype, "sv_perturb ref");
  if (!rc) rc = check_tensor(cand, n, dtype, "sv_perturb cand");
  if (rc) return rc;
  const bool elementwise = op <= SV_OP_SPECIAL_FLIP;
  if (elementwise && op != SV_OP_COPY && !(plan->p >= 0.0 && plan->p <= 1.0))
    return fail(SV_ERR_INVALID_ARG, "sv_perturb: p = %g not in [0, 1]", plan->p);
  const float value = (float)plan->value;
  if ((op == SV_OP_SCALE || op == SV_OP_ADD_AT) && !std::isfinite(value))
    return fail(SV_ERR_INVALID_ARG, "sv_perturb: value = %g is not a finite fp32", plan->value);
  if (!elementwise) {
    if (plan->nidx && !plan->idx) return fail(SV_ERR_INVALID_ARG, "sv_perturb: idx is NULL with nidx > 0");
    for (uint64_t k = 0; k < plan->nidx; ++k)
      if (plan->idx[k] >= n)
        return fail(SV_ERR_INVALID_ARG, "sv_perturb: idx[%llu] = %llu out of range (n = %llu)",
                    (unsigned long long)k, (unsigned long long)plan->idx[k], (unsigned long long)n);
  }
  PerturbParams p;
  std::memset(&p, 0, sizeof p);
  p.k0 = (uint32_t)seed;
  p.k1 = (uint32_t)(seed >> 32);
  p.s0 = (uint32_t)stream_id;
  p.s1 = (uint32_t)(stream_id >> 32);
  p.threshold = width32(plan->p);
  p.value = value;
  p.bits = plan->bits;
  p.op = op;
  DeviceState *ds;
  rc = current_device(&ds);
  if (rc) return rc;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (g_prof_on.load()) {
    e0 = take_event();
    e1 = take_event();
    if (e0) (void)hipEventRecord(e0, t_stream);
  }
  if (elementwise) {
    if (n) SV_HIP(launch_perturb_elementwise(dtype, p, n, ref, cand, ds->cus, t_stream), "perturb kernel launch");
  } else if (plan->nidx) {
    std::lock_guard<std::mutex> lock(ds->mu);
    rc = ensure_pinned(ds->h_idx, ds->h_idx_cap, plan->nidx, "index staging");
    if (!rc) rc = ensure_device(ds->idx, ds->idx_cap, plan->nidx, "index list");
    if (rc) return rc;
    std::memcpy(ds->h_idx, plan->idx, plan->nidx * sizeof(uint64_t));
    SV_HIP(hipMemcpyAsync(ds->idx, ds->h_idx, plan->nidx * sizeof(uint64_t), hipMemcpyHostToDevice, t_stream),
           "index list copy to device");
    SV_HIP(launch_perturb_indexed(dtype, p, ds->idx, plan->nidx, ref, cand, t_stream), "perturb kernel launch");
    SV_HIP(hipStreamSynchronize(t_stream), "hipStreamSynchronize after perturb");
  }
  if (e0 && e1) {
    (void)hipEventRecord(e1, t_stream);
    push_record(SV_PROF_PERTURB, e0, e1);
  }
  return SV_OK;
}

int sv_eval_transform(int32_t which, const uint32_t *in, uint64_t n, uint32_t *out) {
  t_error.clear();
  if (which < SV_EVAL_LN || which > SV_EVAL_F16)
    return fail(SV_ERR_UNSUPPORTED, "sv_eval_transform: unknown transform %d", which);
  int rc = check_tensor(in, n, SV_F32, "sv_eval_transform in");
  if (!rc) rc = check_tensor(out, n, SV_F32, "sv_eval_transform out");
  if (rc || !n) return rc;
  int cus;
  rc = cu_count(&cus);
  if (rc) return rc;
  SV_HIP(launch_eval_transform(which, in, n, out, cus, t_stream), "transform kernel launch");
  return SV_OK;
}

int sv_profile_enable(int32_t on) {
  g_prof_on.store(on ? 1 : 0);
  return SV_OK;
}

int sv_profile_read(int32_t kind, uint64_t *count, double *total_ms) {
  t_error.clear();
  if (!count || !total_ms) return fail(SV_ERR_INVALID_ARG, "sv_profile_read: NULL output");
  std::lock_guard<std::mutex> g(g_prof_mu);
  uint64_t c = 0;
  double tot = 0.0;
  std::vector<ProfRecord> keep;
  int rc = SV_OK;
  for (const ProfRecord &r : g_prof) {
    if (r.kind != kind) {
      keep.push_back(r);
      continue;
    }
    float ms = 0.0f;
    hipError_t e = hipEventSynchronize(r.stop);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess && rc == SV_OK) rc = hip_fail(e, "sv_profile_read");
    tot += ms;
    ++c;
    g_event_pool.push_back(r.start);
    g_event_pool.push_back(r.stop);
  }
  g_prof.swap(keep);
  *count = c;
  *total_ms = tot;
  return rc;
}

int sv_shutdown(void) {
  t_error.clear();
  int prev = 0;
  (void)hipGetDevice(&prev);
  std::lock_guard<std::mutex> g(g_devices_mu);
  for (size_t d = 0; d < g_devices.size(); ++d) {
    DeviceState *s = g_devices[d];
    if (!s) continue;
    std::lock_guard<std::mutex> lock(s->mu);
    (void)hipSetDevice((int)d);
    (void)hipDeviceSynchronize();
    if (s->partials) (void)hipFree(s->partials);
    if (s->table) (void)hipFree(s->table);
    if (s->idx) (void)hipFree(s->idx);
    if (s->h_table) (void)hipHostFree(s->h_table);
    if (s->h_reports) (void)hipHostFree(s->h_reports);
    if (s->h_idx) (void)hipHostFree(s->h_idx);
    if (s->synth_table) (void)hipFree(s->synth_table);
    if (s->h_synth) (void)hipHostFree(s->h_synth);
    if (s->synth_copied) (void)hipEventDestroy(s->synth_copied);
    if (s->synth_done) (void)hipEventDestroy(s->synth_done);
    if (s->counters) (void)hipFree(s->counters);
    if (s->h_done) (void)hipHostFree(s->h_done);
    s->counters = nullptr; s->counters_cap = 0;
    s->h_done = nullptr; s->d_done = nullptr;
    s->synth_table = nullptr; s->h_synth = nullptr; s->synth_copied = nullptr; s->synth_done = nullptr;
    s->synth_table_cap = s->h_synth_cap = 0;
    s->synth_pending = false;
    s->partials = nullptr; s->table = nullptr; s->idx = nullptr;
    s->h_table = nullptr; s->h_reports = nullptr; s->d_reports = nullptr; s->h_idx = nullptr;
    s->partials_cap = s->table_cap = s->idx_cap = 0;
    s->h_table_cap = s->h_reports_cap = s->h_idx_cap = 0;
  }
  perf_shutdown();
  files_shutdown();
  (void)hipSetDevice(prev);
  return SV_OK;
}

}  // extern "C"

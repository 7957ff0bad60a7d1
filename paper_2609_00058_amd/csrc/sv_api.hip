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
// Every check in flight owns a slot: its reports and its completion word in
// host-mapped memory, the pinned staging of its segment table, and what the
// wait needs to finish its reports.  Slots 0 .. SV_MAX_PENDING_CHECKS - 1 hold
// submitted checks; the synchronous calls use the last one.
constexpr int kAsyncSlots = SV_MAX_PENDING_CHECKS;
constexpr int kSyncSlot = kAsyncSlots;
constexpr int kSlots = kAsyncSlots + 1;
constexpr int kDoneStride = 8;        // completion words 64 bytes apart
constexpr int kTicketSeqBits = 56;    // ticket = (device + 1) << 56 | sequence number

struct CheckSlot {
  bool pending = false;          // holds a check not yet waited for
  bool waiting = false;          // a thread waits for it, outside the device lock
  bool launched = false;         // kernels were queued (not when every segment is empty)
  bool stop_at_first = false;
  uint64_t seq = 0;              // the check's sequence number
  hipStream_t stream = nullptr;  // where its kernels were queued
  std::vector<uint64_t> lengths; // n of each segment
  sv_report *h_reports = nullptr;  // pinned, host-mapped, coherent: the finalize writes here
  sv_report *d_reports = nullptr;  // the device address of h_reports
  size_t reports_cap = 0;
  SegDesc *h_table = nullptr;    // pinned staging of the segment table
  size_t h_table_cap = 0;
  bool deferred = false;         // its finalize is left to the next check launched on its stream
  FinalizeArgs fin{};            // ... and what that finalize needs
};

struct DeviceState {
  std::mutex mu;                 // serialises calls that use the scratch below
  int device = 0;
  int cus = 0;
  Partial *partials[2] = {nullptr, nullptr};   // one per (workgroup, segment piece), in two halves that
  size_t partials_cap[2] = {0, 0};              // launched checks take in turn, so that a check can
  int half = 0;                                 // finish the one before it while writing its own (the
                                                // segment tables alternate the same way)
  int deferred = -1;                 // the slot whose finalize waits for the next check on its stream
  SegDesc *table[2] = {nullptr, nullptr};   // batched segment tables, in the halves of the partials
  size_t table_cap[2] = {0, 0};
  std::vector<SegDesc> table_held[2];       // what each device table holds (a repeated batch skips the copy)
  uint64_t *idx = nullptr;
  size_t idx_cap = 0;
  uint64_t *h_idx = nullptr;
  size_t h_idx_cap = 0;
  SynthJob *synth_table = nullptr;   // batched synthesis job table
  size_t synth_table_cap = 0;
  std::vector<SynthJob> synth_held;  // what it holds (a repeated batch skips the copy)
  hipStream_t synth_copy_stream = nullptr;   // where that copy was queued
  SynthJob *h_synth = nullptr;       // its pinned staging
  size_t h_synth_cap = 0;
  hipEvent_t synth_copied = nullptr; // staging -> table copy of the last batch done
  hipEvent_t synth_done = nullptr;   // last batch kernel done (table free to overwrite)
  bool synth_pending = false;        // the two events above have been recorded
  uint32_t *counters = nullptr;      // arrival counters of the check (zero between launches)
  size_t counters_cap = 0;
  uint64_t *firsts = nullptr;        // stop-at-first: a tagged first-mismatch word per segment
  size_t firsts_cap = 0;
  uint64_t firsts_hi = ~0ull;        // seq >> 32 of the launches whose tags the words may hold
  uint64_t *h_done = nullptr;        // pinned, host-mapped, coherent: one completion word per slot
  uint64_t *d_done = nullptr;        // its device address
  uint64_t seq = 0;                  // sequence number of the last check submitted
  CheckSlot slots[kSlots];
  int npending = 0;                  // submitted checks not yet waited for
  bool has_last = false;             // a check has been queued on last_stream
  hipStream_t last_stream = nullptr; // stream of the last check queued
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
    s->device = dev;
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

int ensure_reports(CheckSlot &sl, size_t need) {
  if (need <= sl.reports_cap) return SV_OK;
  const size_t want = std::max(need, sl.reports_cap + sl.reports_cap / 2);
  if (sl.h_reports) (void)hipHostFree(sl.h_reports);
  sl.h_reports = nullptr;
  sl.d_reports = nullptr;
  sl.reports_cap = 0;
  hipError_t e = hipHostMalloc((void **)&sl.h_reports, want * sizeof(sv_report),
                               hipHostMallocMapped | hipHostMallocCoherent);
  if (e != hipSuccess) {
    sl.h_reports = nullptr;
    return fail(SV_ERR_ALLOC, "hipHostMalloc of %zu reports: %s", want, hipGetErrorString(e));
  }
  e = hipHostGetDevicePointer((void **)&sl.d_reports, sl.h_reports, 0);
  if (e != hipSuccess) {
    (void)hipHostFree(sl.h_reports);
    sl.h_reports = nullptr;
    return hip_fail(e, "hipHostGetDevicePointer(reports)");
  }
  sl.reports_cap = want;
  return SV_OK;
}

int ensure_counters(DeviceState *ds, size_t need) {
  if (need <= ds->counters_cap) return SV_OK;
  int rc = ensure_device(ds->counters, ds->counters_cap, need, "arrival counters");
  if (rc) return rc;
  SV_HIP(hipMemset(ds->counters, 0, ds->counters_cap * sizeof(uint32_t)), "hipMemset(arrival counters)");
  return SV_OK;
}

// The stop-at-first words for a check with sequence number seq.  A word's tag
// is the low 32 bits of its launch's sequence number, so a word counts as
// nothing once the tags have moved on -- until they come round again 2^32
// checks later.  The words are therefore cleared (on the calling thread's
// stream, ahead of the check) when they are allocated and whenever the high
// bits of the sequence number differ from those of the last clear.  A zero
// word carries tag 0 and the tile 2^32 - 1, past every tile: it stops nothing.
int ensure_firsts(DeviceState *ds, size_t need, uint64_t seq) {
  if (need > ds->firsts_cap) {
    const int rc = ensure_device(ds->firsts, ds->firsts_cap, need, "first-mismatch words");
    if (rc) return rc;
    ds->firsts_hi = ~0ull;
  }
  if ((seq >> 32) == ds->firsts_hi) return SV_OK;
  const hipError_t e = launch_fill_u64(ds->firsts, ds->firsts_cap, 0, t_stream);
  if (e != hipSuccess) return hip_fail(e, "clearing the first-mismatch words");
  ds->firsts_hi = seq >> 32;
  return SV_OK;
}

int ensure_done(DeviceState *ds) {
  if (ds->h_done) return SV_OK;
  const size_t bytes = (size_t)kSlots * kDoneStride * sizeof(uint64_t);
  hipError_t e = hipHostMalloc((void **)&ds->h_done, bytes, hipHostMallocMapped | hipHostMallocCoherent);
  if (e != hipSuccess) {
    ds->h_done = nullptr;
    return fail(SV_ERR_ALLOC, "hipHostMalloc of the completion words: %s", hipGetErrorString(e));
  }
  e = hipHostGetDevicePointer((void **)&ds->d_done, ds->h_done, 0);
  if (e != hipSuccess) {
    (void)hipHostFree(ds->h_done);
    ds->h_done = nullptr;
    return hip_fail(e, "hipHostGetDevicePointer(completion words)");
  }
  for (int k = 0; k < kSlots * kDoneStride; ++k) ((volatile uint64_t *)ds->h_done)[k] = 0;   // sequence numbers start at 1
  return SV_OK;
}

// Waits until the check with sequence number `seq` has written its reports:
// spins on its host-mapped completion word (a few hundred ns after the
// kernel's last store, well before a stream synchronisation would return),
// asking the stream now and then whether it failed instead.
int wait_done(const volatile uint64_t *flag, uint64_t seq, hipStream_t st) {
  using clock = std::chrono::steady_clock;
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

// floor(p 2^40 / gate) (p 2^40 exact, the quotient rounded to fp64), at most 2^32
uint64_t class_width(double p, uint32_t gate) {
  const uint64_t w = (uint64_t)std::floor(p * 1099511627776.0 / (double)gate);
  return std::min<uint64_t>(w, 1ull << 32);
}

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
  std::memset(&d, 0, sizeof d);      // padding included: tables are compared bytewise
  d.ref = g.ref;
  d.cand = g.cand;
  d.n = g.n;
  d.unit_begin = unit_begin;
  d.rtol = int_dtype(g.dtype) ? 0.0 : g.rtol;
  d.atol = int_dtype(g.dtype) ? 0.0 : g.atol;
  d.dtype = g.dtype;
  d.equal_nan = g.equal_nan ? 1 : 0;
  d.vec_ok = (((uintptr_t)g.ref | (uintptr_t)g.cand) & 15u) == 0 ? 1 : 0;
  d.w0 = d.w1 = 0;
  return d;
}

void zero_report(sv_report *r, uint64_t n) {
  std::memset(r, 0, sizeof *r);
  r->n = n;
  r->first_mismatch = -1;
}

// grid for a check over `units` 16-byte units: at most SV_CMP_BLOCKS_PER_CU
// workgroups per CU, each owning whole waves of units
void compare_grid(uint64_t units, int cus, bool batched, bool stop, uint32_t *nblocks, uint64_t *chunk) {
  const uint64_t per_iter = (uint64_t)kCmpBlock;
  const uint64_t per_cu = stop ? SV_CMP_STOP_BLOCKS_PER_CU : batched ? SV_CMP_BATCH_BLOCKS_PER_CU : SV_CMP_BLOCKS_PER_CU;
  uint64_t nb = std::min<uint64_t>((units + per_iter - 1) / per_iter, (uint64_t)cus * per_cu);
  if (!batched && units <= SV_CMP_FUSE_UNITS) nb = 1;   // small: one workgroup reports by itself
  if (nb == 0) nb = 1;
  uint64_t c = (units + nb - 1) / nb;
  c = (c + kWave - 1) / kWave * kWave;       // whole waves of units per workgroup
  *chunk = c;
  *nblocks = (uint32_t)((units + c - 1) / c);
}

// Queues the finalize that a submitted single-tensor check left to the next
// check on its stream, when that check is not coming: before a wait, a
// readiness query, a check on another stream or a reallocation of scratch.
int flush_deferred(DeviceState *ds) {
  if (ds->deferred < 0) return SV_OK;
  CheckSlot &sl = ds->slots[ds->deferred];
  ds->deferred = -1;
  sl.deferred = false;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (g_prof_on.load()) {
    e0 = take_event();
    e1 = take_event();
    if (e0) (void)hipEventRecord(e0, sl.stream);
  }
  const hipError_t e = launch_finalize(sl.fin, sl.stream);   // its own kernel
  if (e != hipSuccess) return hip_fail(e, "finalize kernel launch");
  if (e0 && e1) {
    (void)hipEventRecord(e1, sl.stream);
    push_record(SV_PROF_FINALIZE, e0, e1);
  }
  return SV_OK;
}

// Waits on the host for every submitted check still pending (they stay
// pending for their waiters).  Called before a check is queued on another
// stream than the previous one and before shared scratch is reallocated, so
// that no queued check can still read what is about to change: a check whose
// completion word has been written has read all of it.
int drain_pending(DeviceState *ds) {
  const int rc = flush_deferred(ds);
  if (rc) return rc;
  if (ds->npending == 0) return SV_OK;
  for (int k = 0; k < kAsyncSlots; ++k) {
    const CheckSlot &sl = ds->slots[k];
    if (!sl.pending || !sl.launched) continue;
    const int rc = wait_done(ds->h_done + (size_t)k * kDoneStride, sl.seq, sl.stream);
    if (rc) return rc;
  }
  return SV_OK;
}

// A validated check: kernel arguments (segment table aside), grid, segments.
struct CheckPlan {
  CompareArgs args;
  uint32_t nblocks = 0;
  const sv_segment *segs = nullptr;   // nullptr: the one segment in args.single
  uint32_t nseg = 0;
  bool stop_at_first = false;
  uint64_t total_units = 0;
};

void plan_single(const sv_segment &g, int cus, CheckPlan &plan) {
  std::memset(&plan.args, 0, sizeof plan.args);
  plan.segs = nullptr;
  plan.nseg = 1;
  plan.stop_at_first = false;
  plan.args.single = make_desc(g, 0);
  plan.args.nseg = 1;
  plan.total_units = plan.args.total_units = units_of(g.dtype, g.n);
  if (plan.total_units) {
    compare_grid(plan.total_units, cus, false, false, &plan.nblocks, &plan.args.chunk);
    plan.args.single.w1 = plan.nblocks - 1;   // its workgroups 0 .. nblocks - 1, slots 0 .. nblocks - 1
  }
}

void plan_batched(const sv_segment *segs, uint32_t nseg, int32_t mode, int cus, CheckPlan &plan) {
  std::memset(&plan.args, 0, sizeof plan.args);
  plan.segs = segs;
  plan.nseg = nseg;
  plan.stop_at_first = mode == SV_CHECK_STOP_AT_FIRST;
  uint64_t total = 0;
  for (uint32_t k = 0; k < nseg; ++k) total += units_of(segs[k].dtype, segs[k].n);
  plan.args.nseg = nseg;
  plan.total_units = plan.args.total_units = total;
  if (total) compare_grid(total, cus, true, plan.stop_at_first, &plan.nblocks, &plan.args.chunk);
  if (total && plan.stop_at_first) {   // workgroups of their own per segment
    uint64_t blocks = 0;
    for (uint32_t k = 0; k < nseg; ++k) blocks += stop_blocks(units_of(segs[k].dtype, segs[k].n), plan.args.chunk);
    plan.nblocks = blocks <= kMaxStopBlocks ? (uint32_t)blocks : 0;   // 0: too many, refused at submission
  }
}

// Queues the kernels of `plan` into slot k on the selected stream and marks
// the slot pending under a new sequence number.  The check kernel and its
// finalize write the reports into the slot's host-mapped memory, then the
// sequence number into the slot's completion word; a submitted check leaves
// its finalize to the next check on its stream (see below).
int submit_check(DeviceState *ds, int k, CheckPlan &plan) {
  hipStream_t st = t_stream;
  CheckSlot &sl = ds->slots[k];
  const uint32_t nseg = plan.nseg;
  const bool batched = plan.segs != nullptr;
  sl.lengths.resize(nseg);
  for (uint32_t j = 0; j < nseg; ++j) sl.lengths[j] = batched ? plan.segs[j].n : plan.args.single.n;
  sl.stop_at_first = plan.stop_at_first;
  sl.launched = false;
  sl.waiting = false;
  if (plan.total_units == 0) {                   // nothing to launch: every report is empty
    sl.seq = ++ds->seq;
    sl.pending = true;
    return SV_OK;
  }
  if (plan.nblocks == 0)
    return fail(SV_ERR_INVALID_ARG, "stop-at-first check of %u segments: more than %u workgroups", nseg,
                (unsigned)kMaxStopBlocks);
  const size_t nfirsts = plan.stop_at_first ? (size_t)nseg * kFirstStride : 0;
  const int par = ds->half;                      // this check's half of the partials
  const bool grow = (size_t)plan.nblocks + nseg > ds->partials_cap[par] ||
                    (batched && nseg > ds->table_cap[par]) || nfirsts > ds->firsts_cap;
  int rc = SV_OK;
  if (grow || (ds->has_last && ds->last_stream != st)) rc = drain_pending(ds);
  if (!rc) rc = ensure_device(ds->partials[par], ds->partials_cap[par], (size_t)plan.nblocks + nseg, "partials");
  if (!rc && nfirsts) rc = ensure_firsts(ds, nfirsts, ds->seq + 1);
  if (!rc && batched && nseg > ds->table_cap[par]) {
    ds->table_held[par].clear();               // a new allocation holds nothing yet
    rc = ensure_device(ds->table[par], ds->table_cap[par], nseg, "segment table");
  }
  if (!rc && batched) rc = ensure_pinned(sl.h_table, sl.h_table_cap, nseg, "segment table staging");
  if (!rc) rc = ensure_reports(sl, nseg);
  if (!rc) rc = ensure_counters(ds, 1);
  if (!rc) rc = ensure_done(ds);
  if (rc) return rc;
  CompareArgs &args = plan.args;
  if (batched) {
    uint64_t begin = 0, blk = 0;
    for (uint32_t j = 0; j < nseg; ++j) {
      SegDesc &d = sl.h_table[j];
      d = make_desc(plan.segs[j], begin);
      const uint64_t units = units_of(plan.segs[j].dtype, plan.segs[j].n);
      if (plan.stop_at_first) {
        d.w0 = (uint32_t)blk;
        blk += stop_blocks(units, plan.args.chunk);
        d.w1 = (uint32_t)(blk - (units ? 1 : 0));
      } else if (units) {
        d.w0 = (uint32_t)(begin / plan.args.chunk);
        d.w1 = (uint32_t)((begin + units - 1) / plan.args.chunk);
      }
      begin += units;
    }
    // the same batch as the last one in this half (a check repeated on the same
    // tensors) finds its table in place: only this call writes the device table
    std::vector<SegDesc> &held = ds->table_held[par];
    if (held.size() != nseg || std::memcmp(held.data(), sl.h_table, nseg * sizeof(SegDesc)) != 0) {
      SV_HIP(hipMemcpyAsync(ds->table[par], sl.h_table, nseg * sizeof(SegDesc), hipMemcpyHostToDevice, st),
             "segment table copy to device");
      held.assign(sl.h_table, sl.h_table + nseg);
    }
    args.segs = ds->table[par];
  }
  args.stop_at_first = plan.stop_at_first ? 1 : 0;
  args.firsts = ds->firsts;
  args.fused = batched ? 0 : plan.nblocks == 1 ? 1 : plan.nblocks <= SV_CMP_LAST_BLOCK_MAX ? 2 : 0;
  args.partials = ds->partials[par];
  args.counter = ds->counters;
  args.reports = sl.d_reports;
  args.done = ds->d_done + (size_t)k * kDoneStride;
  args.seq = ds->seq + 1;
  const bool defer = !args.fused && k != kSyncSlot;   // see below
  hipEvent_t e0 = nullptr, e1 = nullptr, e2 = nullptr;
  if (g_prof_on.load()) {
    e0 = take_event();
    e1 = take_event();
    if (!args.fused && !defer) e2 = take_event();
    if (e0) (void)hipEventRecord(e0, st);
  }
  uint32_t mask = 0;
  for (uint32_t j = 0; j < nseg; ++j) {
    const uint64_t n = batched ? plan.segs[j].n : args.single.n;
    if (n) mask |= 1u << (batched ? plan.segs[j].dtype : args.single.dtype);
  }
  // A submitted check leaves its finalize to the next check on its stream,
  // whose first workgroups run it (one launch less per check when checks
  // follow each other).  A check with a grid of its own takes it on; a
  // one-workgroup check (which reports by itself) and a stop-at-first check
  // have it queued first.
  args.nprev = 0;
  args.prev = FinalizeArgs{};
  if (ds->deferred >= 0) {
    CheckSlot &pd = ds->slots[ds->deferred];
    if (args.fused == 0 && !args.stop_at_first && pd.stream == st) {
      args.prev = pd.fin;
      args.nprev = pd.fin.nseg;
      ds->deferred = -1;
      pd.deferred = false;
    } else if ((rc = flush_deferred(ds)) != SV_OK) {
      return rc;
    }
  }
  hipError_t e = launch_compare(args, plan.nblocks + args.nprev, mask, st);
  if (e != hipSuccess) return hip_fail(e, "check kernel launch");
  if (e1) (void)hipEventRecord(e1, st);
  if (defer) {
    sl.fin = finalize_args(args);
    sl.deferred = true;
    ds->deferred = k;
  } else if (!args.fused) {
    e = launch_finalize(finalize_args(args), st);
    if (e != hipSuccess) return hip_fail(e, "finalize kernel launch");
  }
  ds->seq = args.seq;
  ds->half ^= 1;
  ds->has_last = true;
  ds->last_stream = st;
  sl.seq = args.seq;
  sl.stream = st;
  sl.launched = true;
  sl.pending = true;
  if (e0 && e1) {
    push_record(SV_PROF_COMPARE, e0, e1);
    if (e2) {
      (void)hipEventRecord(e2, st);
      push_record(SV_PROF_FINALIZE, e1, e2);
    }
  }
  return SV_OK;
}

// The reports of a completed check, out of its slot.  Segments with no
// elements get their empty report here; in stop-at-first mode a failing
// segment keeps only its verdict and its first index.
void finish_check(const CheckSlot &sl, sv_report *out) {
  for (size_t j = 0; j < sl.lengths.size(); ++j) {
    const uint64_t n = sl.lengths[j];
    if (n)
      out[j] = sl.h_reports[j];
    else
      zero_report(&out[j], 0);
    if (sl.stop_at_first && out[j].mismatches) {
      const int64_t first = out[j].first_mismatch;
      zero_report(&out[j], n);
      out[j].mismatches = 1;
      out[j].first_mismatch = first;
    }
  }
}

// A synchronous check: submit into the synchronous slot and wait (the
// caller holds the device lock throughout).
int run_sync(DeviceState *ds, CheckPlan &plan, sv_report *out) {
  CheckSlot &sl = ds->slots[kSyncSlot];
  int rc = submit_check(ds, kSyncSlot, plan);
  if (!rc && sl.launched) rc = wait_done(ds->h_done + (size_t)kSyncSlot * kDoneStride, sl.seq, sl.stream);
  if (!rc) finish_check(sl, out);
  sl.pending = false;
  return rc;
}

uint64_t make_ticket(int device, uint64_t seq) { return ((uint64_t)(device + 1) << kTicketSeqBits) | seq; }

// The device state a ticket names, or nullptr.
DeviceState *ticket_device(uint64_t ticket) {
  const uint64_t d = ticket >> kTicketSeqBits;
  std::lock_guard<std::mutex> g(g_devices_mu);
  if (d == 0 || d > g_devices.size()) return nullptr;
  return g_devices[d - 1];
}

// The async slot holding `ticket`, or -1 (caller holds the device lock).
int ticket_slot(const DeviceState *ds, uint64_t ticket) {
  const uint64_t seq = ticket & ((1ull << kTicketSeqBits) - 1);
  for (int k = 0; k < kAsyncSlots; ++k)
    if (ds->slots[k].pending && ds->slots[k].seq == seq) return k;
  return -1;
}

// A free async slot for a submission, or an error (caller holds the lock).
int take_slot(DeviceState *ds, int *k) {
  for (int j = 0; j < kAsyncSlots; ++j)
    if (!ds->slots[j].pending) {
      *k = j;
      return SV_OK;
    }
  return fail(SV_ERR_INVALID_ARG, "%d checks are already pending on device %d: wait for one first",
              kAsyncSlots, ds->device);
}

// Validates the arguments of one synthesis and prepares its kernel
// parameters; issues no HIP call.
int prepare_synth(uint64_t seed, uint64_t stream_id, int32_t dtype, int32_t dist, const sv_dist_params *params,
                  uint64_t n, void *out, SynthParams *pp) {
  if (!valid_dtype(dtype)) return fail(SV_ERR_UNSUPPORTED, "sv_synth: unknown dtype %d", dtype);
  if (dist < SV_UNIFORM || dist > SV_PERMUTATION) return fail(SV_ERR_UNSUPPORTED, "sv_synth: unknown dist %d", dist);
  if ((dist == SV_INT_RANGE || dist == SV_PERMUTATION) != int_dtype(dtype))
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
      // S / 256 of the elements (S = ceil(256 tot)) are candidates; among them each
      // class takes a width floor(p 2^32 256 / S) of the class word, cumulative
      p.gate = (uint32_t)std::ceil(256.0 * tot);
      if (p.gate) {
        const uint64_t full = 1ull << 32;
        p.t_nan = class_width(params->p_nan, p.gate);
        p.t_inf = std::min(full, p.t_nan + class_width(params->p_inf, p.gate));
        p.t_den = std::min(full, p.t_inf + class_width(params->p_denorm, p.gate));
        p.t_zero = std::min(full, p.t_den + class_width(params->p_zero, p.gate));
      }
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
    if (dist == SV_PERMUTATION) {
      if (p.range == 0 || p.range > (1ull << 60))
        return fail(SV_ERR_INVALID_ARG, "sv_synth: a permutation takes at most 2^60 values");
      if (n > p.range)
        return fail(SV_ERR_INVALID_ARG, "sv_synth: %llu elements exceed the %llu values of the permutation",
                    (unsigned long long)n, (unsigned long long)p.range);
      uint32_t bits = 0;                          // smallest b with 2^b >= N
      while ((1ull << bits) < p.range) ++bits;
      p.half = bits < 2 ? 1u : (bits + 1u) / 2u;
    }
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

// ------------------------------------------------------------ sv_compare_noalloc
// The single-tensor check with its scratch in a fixed device array instead of
// memory the library allocates: the workgroup partials, the arrival counter,
// the report and the completion word that the check kernel and its finalize
// write.  The array is a host-side stand-in in host code: its device address
// on each GPU comes from hipGetSymbolAddress, taken once per device with that
// device current, and only that address is handed to kernels and copies.
constexpr size_t kNaPartials = 4096;            // workgroup partials the array holds
constexpr size_t kNaCounterOff = 0;             // uint32 arrival counter (zero between launches)
constexpr size_t kNaDoneOff = 64;               // uint64 completion word
constexpr size_t kNaReportOff = 128;            // sv_report
constexpr size_t kNaPartialsOff = 256;
constexpr size_t kNaBytes = kNaPartialsOff + kNaPartials * sizeof(Partial);
static_assert(kNaReportOff + sizeof(sv_report) <= kNaPartialsOff, "scratch layout");
constexpr int kNaMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kNaBytes];

namespace {
struct NoAllocDevice {
  std::mutex mu;                 // one check at a time per device: they share the array
  bool ready = false;
  unsigned char *ptr = nullptr;  // device address of `scratch` on this device
  int cus = 0;
};
NoAllocDevice g_noalloc[kNaMaxDevices];

// Set-up on the current device (first call there): the array's device
// address and the CU count.  The caller holds d.mu.
int noalloc_setup(NoAllocDevice &d, int dev) {
  if (d.ready) return SV_OK;
  void *p = nullptr;
  SV_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
  int cus = 0;
  SV_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev),
         "hipDeviceGetAttribute(multiProcessorCount)");
  d.ptr = (unsigned char *)p;
  d.cus = cus > 0 ? cus : 1;
  d.ready = true;
  return SV_OK;
}
}  // namespace

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
  if (dist == SV_PERMUTATION && (offset > p.range || n > p.range - offset))
    return fail(SV_ERR_INVALID_ARG, "sv_synth_window: elements [%llu, %llu) lie past the %llu values of the permutation",
                (unsigned long long)offset, (unsigned long long)(offset + n), (unsigned long long)p.range);
  const uint64_t per_block =
      dist == SV_PERMUTATION ? 1
      : ((dist == SV_INT_RANGE && dtype != SV_U8) || (dist == SV_UNIFORM && dtype == SV_F64)) ? 2
      : (dist == SV_UNIFORM && dtype == SV_BF16)                                              ? 8
                                                                                            : 4;
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
  uint64_t total_vecs = 0;
  for (uint32_t k = 0; k < njobs; ++k) {
    const sv_synth_job &j = jobs[k];
    int rc = prepare_synth(j.seed, j.stream_id, j.dtype, j.dist, &j.params, j.n, j.out, &params[k]);
    if (rc) {
      t_error = "job " + std::to_string(k) + ": " + t_error;
      return rc;
    }
    if (!j.n) continue;
    if (!table_kind(j.dtype) || j.dist == SV_PERMUTATION) {
      direct_jobs.push_back(k);
      continue;
    }
    table_jobs.push_back(k);
    total_vecs += units_of(j.dtype, j.n);
  }
  if (table_jobs.empty() && direct_jobs.empty()) return SV_OK;
  DeviceState *ds;
  int rc = current_device(&ds);
  if (rc) return rc;
  const uint32_t rounds = synth_tile_rounds(total_vecs, ds->cus);   // vectors per thread in a tile
  const uint64_t tile_vecs = (uint64_t)rounds * kBlock;
  uint64_t tiles = 0;
  std::lock_guard<std::mutex> lock(ds->mu);
  hipStream_t st = t_stream;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (g_prof_on.load()) {
    e0 = take_event();
    e1 = take_event();
  }
  const uint32_t nt = (uint32_t)table_jobs.size();
  if (nt) {
    std::vector<SynthJob> table(nt);
    uint64_t begin = 0;
    for (uint32_t t = 0; t < nt; ++t) {
      const sv_synth_job &j = jobs[table_jobs[t]];
      SynthJob &d = table[t];
      std::memset(&d, 0, sizeof d);
      d.p = params[table_jobs[t]];
      d.out = j.out;
      d.n = j.n;
      d.nvec = units_of(j.dtype, j.n);
      d.tile_begin = begin;
      d.kind = j.dist * 4 + j.dtype;
      d.vec_ok = ((uintptr_t)j.out & 15u) == 0 ? 1 : 0;
      begin += (d.nvec + tile_vecs - 1) / tile_vecs;
    }
    tiles = begin;
    // the same batch as the last one (synthesis repeated into the same tensors)
    // finds its table in place: only this call writes the device table
    const bool same = ds->synth_held.size() == nt &&
                      std::memcmp(ds->synth_held.data(), table.data(), nt * sizeof(SynthJob)) == 0;
    if (same && st != ds->synth_copy_stream)       // that copy may still be queued on another stream
      SV_HIP(hipStreamWaitEvent(st, ds->synth_copied, 0), "order after the job-table copy");
    if (!same) {
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
      ds->synth_held.clear();
      rc = ensure_pinned(ds->h_synth, ds->h_synth_cap, nt, "job table staging");
      if (!rc) rc = ensure_device(ds->synth_table, ds->synth_table_cap, nt, "job table");
      if (rc) return rc;
      std::memcpy(ds->h_synth, table.data(), nt * sizeof(SynthJob));
      SV_HIP(hipMemcpyAsync(ds->synth_table, ds->h_synth, nt * sizeof(SynthJob), hipMemcpyHostToDevice, st),
             "job table copy to device");
      SV_HIP(hipEventRecord(ds->synth_copied, st), "hipEventRecord");
      ds->synth_held.swap(table);
      ds->synth_copy_stream = st;
    }
  }
  if (e0) (void)hipEventRecord(e0, st);
  if (nt)
    SV_HIP(launch_synth_batched(ds->synth_table, nt, tiles, rounds, ds->cus, st), "batched synthesis kernel launch");
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
  CheckPlan plan;
  plan_single(g, ds->cus, plan);
  return run_sync(ds, plan, report);
}

int sv_compare_batched(const sv_segment *segs, uint32_t nseg, sv_report *reports) {
  return sv_compare_batched_mode(segs, nseg, SV_CHECK_FULL, reports);
}

// Arguments of a batched check; no HIP call.
static int check_batch(const sv_segment *segs, uint32_t nseg, int32_t mode, const char *who) {
  if (mode != SV_CHECK_FULL && mode != SV_CHECK_STOP_AT_FIRST)
    return fail(SV_ERR_UNSUPPORTED, "%s: unknown mode %d", who, mode);
  if (nseg && !segs) return fail(SV_ERR_INVALID_ARG, "%s: segs is NULL", who);
  for (uint32_t k = 0; k < nseg; ++k) {
    int rc = check_seg(segs[k], k);
    if (rc) return rc;
  }
  return SV_OK;
}

int sv_compare_batched_mode(const sv_segment *segs, uint32_t nseg, int32_t mode, sv_report *reports) {
  t_error.clear();
  if (mode != SV_CHECK_FULL && mode != SV_CHECK_STOP_AT_FIRST)
    return fail(SV_ERR_UNSUPPORTED, "sv_compare_batched_mode: unknown mode %d", mode);
  if (nseg == 0) return SV_OK;
  if (!segs || !reports) return fail(SV_ERR_INVALID_ARG, "sv_compare_batched: segs or reports is NULL");
  int rc = check_batch(segs, nseg, mode, "sv_compare_batched");
  if (rc) return rc;
  uint64_t total = 0;
  for (uint32_t k = 0; k < nseg; ++k) total += units_of(segs[k].dtype, segs[k].n);
  if (total == 0) {
    for (uint32_t k = 0; k < nseg; ++k) zero_report(&reports[k], 0);
    return SV_OK;
  }
  DeviceState *ds;
  rc = current_device(&ds);
  if (rc) return rc;
  std::lock_guard<std::mutex> lock(ds->mu);
  CheckPlan plan;
  plan_batched(segs, nseg, mode, ds->cus, plan);
  return run_sync(ds, plan, reports);
}

int sv_compare_submit(const void *ref, const void *cand, uint64_t n, int32_t dtype, double rtol, double atol,
                      int32_t equal_nan, uint64_t *ticket) {
  t_error.clear();
  if (!ticket) return fail(SV_ERR_INVALID_ARG, "sv_compare_submit: ticket is NULL");
  const sv_segment g{ref, cand, n, dtype, rtol, atol, equal_nan};
  int rc = check_seg(g, 0);
  if (rc) return rc;
  DeviceState *ds;
  rc = current_device(&ds);
  if (rc) return rc;
  std::lock_guard<std::mutex> lock(ds->mu);
  int k;
  rc = take_slot(ds, &k);
  if (rc) return rc;
  CheckPlan plan;
  plan_single(g, ds->cus, plan);
  rc = submit_check(ds, k, plan);
  if (rc) {
    ds->slots[k].pending = false;
    return rc;
  }
  ++ds->npending;
  *ticket = make_ticket(ds->device, ds->slots[k].seq);
  return SV_OK;
}

int sv_compare_batched_submit(const sv_segment *segs, uint32_t nseg, int32_t mode, uint64_t *ticket) {
  t_error.clear();
  if (!ticket) return fail(SV_ERR_INVALID_ARG, "sv_compare_batched_submit: ticket is NULL");
  int rc = check_batch(segs, nseg, mode, "sv_compare_batched_submit");
  if (rc) return rc;
  DeviceState *ds;
  rc = current_device(&ds);
  if (rc) return rc;
  std::lock_guard<std::mutex> lock(ds->mu);
  int k;
  rc = take_slot(ds, &k);
  if (rc) return rc;
  CheckPlan plan;
  plan_batched(segs, nseg, mode, ds->cus, plan);
  rc = submit_check(ds, k, plan);
  if (rc) {
    ds->slots[k].pending = false;
    return rc;
  }
  ++ds->npending;
  *ticket = make_ticket(ds->device, ds->slots[k].seq);
  return SV_OK;
}

int sv_compare_ready(uint64_t ticket, int32_t *ready) {
  t_error.clear();
  if (!ready) return fail(SV_ERR_INVALID_ARG, "sv_compare_ready: ready is NULL");
  DeviceState *ds = ticket_device(ticket);
  if (!ds) return fail(SV_ERR_INVALID_ARG, "sv_compare_ready: ticket %#llx names no device in use",
                       (unsigned long long)ticket);
  std::lock_guard<std::mutex> lock(ds->mu);
  const int k = ticket_slot(ds, ticket);
  if (k < 0) return fail(SV_ERR_INVALID_ARG, "sv_compare_ready: ticket %#llx is not pending", (unsigned long long)ticket);
  const CheckSlot &sl = ds->slots[k];
  const volatile uint64_t *flag = ds->h_done + (size_t)k * kDoneStride;
  if (sl.deferred) {
    const int rc = flush_deferred(ds);
    if (rc) return rc;
  }
  if (!sl.launched || *flag == sl.seq) {
    *ready = 1;
    return SV_OK;
  }
  const hipError_t e = hipStreamQuery(sl.stream);
  if (e != hipSuccess && e != hipErrorNotReady) return hip_fail(e, "sv_compare_ready");
  if (e == hipSuccess && *flag != sl.seq)
    return fail(SV_ERR_HIP, "the check kernel finished without writing its reports");
  *ready = *flag == sl.seq ? 1 : 0;
  return SV_OK;
}

int sv_compare_wait(uint64_t ticket, sv_report *reports, uint32_t nreports) {
  t_error.clear();
  DeviceState *ds = ticket_device(ticket);
  if (!ds) return fail(SV_ERR_INVALID_ARG, "sv_compare_wait: ticket %#llx names no device in use",
                       (unsigned long long)ticket);
  int k;
  uint64_t seq;
  bool launched;
  hipStream_t st;
  {
    std::lock_guard<std::mutex> lock(ds->mu);
    k = ticket_slot(ds, ticket);
    if (k < 0 || ds->slots[k].waiting)
      return fail(SV_ERR_INVALID_ARG, "sv_compare_wait: ticket %#llx is not pending (already waited for?)",
                  (unsigned long long)ticket);
    CheckSlot &sl = ds->slots[k];
    if (nreports != sl.lengths.size())
      return fail(SV_ERR_INVALID_ARG, "sv_compare_wait: the check has %zu reports, nreports = %u",
                  sl.lengths.size(), nreports);
    if (nreports && !reports) return fail(SV_ERR_INVALID_ARG, "sv_compare_wait: reports is NULL");
    if (sl.deferred) {
      const int rc = flush_deferred(ds);
      if (rc) return rc;
    }
    sl.waiting = true;
    seq = sl.seq;
    launched = sl.launched;
    st = sl.stream;
  }
  // the slot stays pending (not reusable) while this thread spins unlocked
  const int rc = launched ? wait_done(ds->h_done + (size_t)k * kDoneStride, seq, st) : SV_OK;
  std::lock_guard<std::mutex> lock(ds->mu);
  CheckSlot &sl = ds->slots[k];
  if (!rc) finish_check(sl, reports);
  sl.pending = false;
  sl.waiting = false;
  --ds->npending;
  return rc;
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
  if (which < SV_EVAL_LN || which > SV_EVAL_BF16)
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

int sv_testing_set_sequence(uint64_t last) {
  t_error.clear();
  if (last >= (1ull << kTicketSeqBits) - (1ull << 32))
    return fail(SV_ERR_INVALID_ARG, "sv_testing_set_sequence: %llu is too large", (unsigned long long)last);
  DeviceState *ds;
  int rc = current_device(&ds);
  if (rc) return rc;
  std::lock_guard<std::mutex> lock(ds->mu);
  if (ds->npending)
    return fail(SV_ERR_INVALID_ARG, "sv_testing_set_sequence: %d submitted checks not yet waited for", ds->npending);
  ds->seq = last;
  // numbers may repeat: no completion word may still hold one of them (none is
  // pending, so the host may write them), and the next stop-at-first check
  // clears the tagged words
  if (ds->h_done)
    for (int k = 0; k < kSlots; ++k) ds->h_done[(size_t)k * kDoneStride] = ~0ull;
  ds->firsts_hi = ~0ull;
  return SV_OK;
}

int sv_compare_noalloc(const void *ref, const void *cand, uint64_t n, int32_t dtype, double rtol, double atol,
                       int32_t equal_nan, sv_report *report) {
  t_error.clear();
  if (!report) return fail(SV_ERR_INVALID_ARG, "sv_compare_noalloc: report is NULL");
  const sv_segment g{ref, cand, n, dtype, rtol, atol, equal_nan};
  int rc = check_seg(g, 0);
  if (rc) return rc;
  if (!n) {
    zero_report(report, 0);
    return SV_OK;
  }
  int dev = 0;
  SV_HIP(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= kNaMaxDevices)
    return fail(SV_ERR_UNSUPPORTED, "sv_compare_noalloc: device %d beyond the %d it keeps scratch for", dev,
                kNaMaxDevices);
  NoAllocDevice &d = g_noalloc[dev];
  std::lock_guard<std::mutex> lock(d.mu);
  rc = noalloc_setup(d, dev);
  if (rc) return rc;
  CheckPlan plan;
  plan_single(g, d.cus, plan);
  if ((size_t)plan.nblocks + 1 > kNaPartials)
    return fail(SV_ERR_UNSUPPORTED, "sv_compare_noalloc: the check needs %u workgroup partials, the fixed scratch "
                "holds %zu", plan.nblocks + 1, kNaPartials);
  hipStream_t st = t_stream;
  CompareArgs &args = plan.args;
  args.stop_at_first = 0;
  args.firsts = nullptr;
  args.fused = plan.nblocks == 1 ? 1 : plan.nblocks <= SV_CMP_LAST_BLOCK_MAX ? 2 : 0;
  args.partials = (Partial *)(d.ptr + kNaPartialsOff);
  args.counter = (uint32_t *)(d.ptr + kNaCounterOff);
  args.reports = (sv_report *)(d.ptr + kNaReportOff);
  args.done = (uint64_t *)(d.ptr + kNaDoneOff);
  args.seq = 1;
  args.nprev = 0;
  args.prev = FinalizeArgs{};
  // the arrival counter must start at zero: cleared by a kernel (the 8-byte
  // word holding it), not a memset, before every check
  SV_HIP(launch_fill_u64((uint64_t *)(d.ptr + kNaCounterOff), 1, 0, st), "clearing the arrival counter");
  SV_HIP(launch_compare(args, plan.nblocks, 1u << dtype, st), "check kernel launch");
  if (!args.fused) SV_HIP(launch_finalize(finalize_args(args), st), "finalize kernel launch");
  SV_HIP(hipMemcpyAsync(report, d.ptr + kNaReportOff, sizeof(sv_report), hipMemcpyDeviceToHost, st),
         "report copy to host");
  SV_HIP(hipStreamSynchronize(st), "waiting for the check");
  return SV_OK;
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
    for (int h = 0; h < 2; ++h) {
      if (s->partials[h]) (void)hipFree(s->partials[h]);
      s->partials[h] = nullptr;
      s->partials_cap[h] = 0;
    }
    s->deferred = -1;
    s->half = 0;
    for (int h = 0; h < 2; ++h) {
      if (s->table[h]) (void)hipFree(s->table[h]);
      s->table[h] = nullptr;
      s->table_cap[h] = 0;
      s->table_held[h].clear();
    }
    s->synth_held.clear();
    s->synth_copy_stream = nullptr;
    if (s->idx) (void)hipFree(s->idx);
    for (CheckSlot &sl : s->slots) {
      if (sl.h_reports) (void)hipHostFree(sl.h_reports);
      if (sl.h_table) (void)hipHostFree(sl.h_table);
      sl = CheckSlot();
    }
    s->npending = 0;
    s->has_last = false;
    s->last_stream = nullptr;
    if (s->h_idx) (void)hipHostFree(s->h_idx);
    if (s->synth_table) (void)hipFree(s->synth_table);
    if (s->h_synth) (void)hipHostFree(s->h_synth);
    if (s->synth_copied) (void)hipEventDestroy(s->synth_copied);
    if (s->synth_done) (void)hipEventDestroy(s->synth_done);
    if (s->counters) (void)hipFree(s->counters);
    if (s->firsts) (void)hipFree(s->firsts);
    s->firsts = nullptr; s->firsts_cap = 0; s->firsts_hi = ~0ull;
    if (s->h_done) (void)hipHostFree(s->h_done);
    s->counters = nullptr; s->counters_cap = 0;
    s->h_done = nullptr; s->d_done = nullptr;
    s->synth_table = nullptr; s->h_synth = nullptr; s->synth_copied = nullptr; s->synth_done = nullptr;
    s->synth_table_cap = s->h_synth_cap = 0;
    s->synth_pending = false;
    s->idx = nullptr;
    s->h_idx = nullptr;
    s->idx_cap = 0;
    s->h_idx_cap = 0;
  }
  perf_shutdown();
  files_shutdown();
  (void)hipSetDevice(prev);
  return SV_OK;
}

}  // extern "C"

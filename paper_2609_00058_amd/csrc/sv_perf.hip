// sv_perf.hip -- the performance stage and the reward (sv_kernel_load,
// sv_kernel_launch, sv_kernel_time, sv_reward): Eq. (3) and Eq. (4).
//
// A candidate arrives as a gfx950 code object and is launched through the
// module API with its arguments packed into one buffer.  Each timed run is
// bracketed by HIP events on the caller's stream; an optional fill of library
// scratch before each run (outside the events) evicts the L2s and the Infinity
// Cache, so every run starts cold.  The events of a call are kept per device
// and reused.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <mutex>
#include <new>
#include <vector>

#include "sv_internal.h"

struct sv_kernel {
  hipModule_t module;
  hipFunction_t fn;
  int device;
};

namespace sv {
namespace {

constexpr uint32_t kMaxReps = 1u << 20;
constexpr uint64_t kMaxFlush = 1ull << 34;

struct PerfState {
  std::mutex mu;
  uint4 *flush = nullptr;
  size_t flush_cap = 0;                 // bytes
  std::vector<hipEvent_t> events;
};

std::mutex g_perf_mu;
std::vector<PerfState *> g_perf;

PerfState *perf_state(int dev) {
  std::lock_guard<std::mutex> g(g_perf_mu);
  if ((size_t)dev >= g_perf.size()) g_perf.resize(dev + 1, nullptr);
  if (!g_perf[dev]) g_perf[dev] = new PerfState;
  return g_perf[dev];
}

// Plain streaming stores of zeros over the flush buffer.
__global__ __launch_bounds__(kBlock) void fill_kernel(uint4 *p, uint64_t n) {
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride) p[i] = make_uint4(0, 0, 0, 0);
}

bool looks_like_code_object(const void *p, uint64_t size) {
  static const char kBundle[] = "__CLANG_OFFLOAD_BUNDLE__";
  const unsigned char *b = (const unsigned char *)p;
  if (size >= 4 && b[0] == 0x7F && b[1] == 'E' && b[2] == 'L' && b[3] == 'F') return true;
  return size >= sizeof kBundle - 1 && std::memcmp(p, kBundle, sizeof kBundle - 1) == 0;
}

int check_launch(const sv_kernel *k, const sv_launch *l) {
  if (!k || !l) return api_fail(SV_ERR_INVALID_ARG, "sv_kernel: kernel or launch is NULL");
  uint64_t threads = 1;
  for (int d = 0; d < 3; ++d) {
    if (l->grid[d] == 0 || l->block[d] == 0)
      return api_fail(SV_ERR_INVALID_ARG, "sv_kernel: grid and block dimensions must be >= 1");
    threads *= l->block[d];
  }
  if (threads > 1024) return api_fail(SV_ERR_INVALID_ARG, "sv_kernel: more than 1024 threads per workgroup");
  if (l->args_size && !l->args) return api_fail(SV_ERR_INVALID_ARG, "sv_kernel: args is NULL with args_size > 0");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return api_hip_fail(e, "hipGetDevice");
  if (dev != k->device) return api_fail(SV_ERR_INVALID_ARG, "sv_kernel: the kernel was loaded on another device");
  return SV_OK;
}

hipError_t launch_once(const sv_kernel *k, const sv_launch *l, hipStream_t st) {
  size_t size = l->args_size;
  void *extra[] = {HIP_LAUNCH_PARAM_BUFFER_POINTER, const_cast<void *>(l->args), HIP_LAUNCH_PARAM_BUFFER_SIZE,
                   &size, HIP_LAUNCH_PARAM_END};
  return hipModuleLaunchKernel(k->fn, l->grid[0], l->grid[1], l->grid[2], l->block[0], l->block[1], l->block[2],
                               l->shared_bytes, st, nullptr, size ? extra : nullptr);
}

}  // namespace

void perf_shutdown() {
  std::lock_guard<std::mutex> g(g_perf_mu);
  for (PerfState *ps : g_perf) {
    if (!ps) continue;
    std::lock_guard<std::mutex> lock(ps->mu);
    if (ps->flush) (void)hipFree(ps->flush);
    ps->flush = nullptr;
    ps->flush_cap = 0;
    for (hipEvent_t e : ps->events) (void)hipEventDestroy(e);
    ps->events.clear();
  }
}

}  // namespace sv

using namespace sv;

extern "C" {

int sv_kernel_load(const void *code_object, uint64_t size, const char *name, sv_kernel **out) {
  api_clear_error();
  if (!code_object || !size || !name || !out)
    return api_fail(SV_ERR_INVALID_ARG, "sv_kernel_load: NULL argument or empty code object");
  if (!looks_like_code_object(code_object, size))
    return api_fail(SV_ERR_INVALID_ARG, "sv_kernel_load: not an ELF code object or offload bundle");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return api_hip_fail(e, "hipGetDevice");
  hipModule_t m = nullptr;
  e = hipModuleLoadData(&m, code_object);
  if (e != hipSuccess) return api_hip_fail(e, "hipModuleLoadData");
  hipFunction_t f = nullptr;
  e = hipModuleGetFunction(&f, m, name);
  if (e != hipSuccess) {
    (void)hipModuleUnload(m);
    return api_hip_fail(e, "hipModuleGetFunction");
  }
  sv_kernel *k = new (std::nothrow) sv_kernel{m, f, dev};
  if (!k) {
    (void)hipModuleUnload(m);
    return api_fail(SV_ERR_ALLOC, "sv_kernel_load: out of host memory");
  }
  *out = k;
  return SV_OK;
}

int sv_kernel_free(sv_kernel *k) {
  api_clear_error();
  if (!k) return SV_OK;
  hipError_t e = hipModuleUnload(k->module);
  delete k;
  return e == hipSuccess ? SV_OK : api_hip_fail(e, "hipModuleUnload");
}

int sv_kernel_launch(const sv_kernel *k, const sv_launch *launch) {
  api_clear_error();
  int rc = check_launch(k, launch);
  if (rc) return rc;
  hipError_t e = launch_once(k, launch, api_stream());
  return e == hipSuccess ? SV_OK : api_hip_fail(e, "candidate launch");
}

int sv_kernel_time(const sv_kernel *k, const sv_launch *launch, uint32_t warmup, uint32_t reps,
                   uint64_t flush_bytes, float *rep_ms, sv_timing *out) {
  api_clear_error();
  int rc = check_launch(k, launch);
  if (rc) return rc;
  if (!out) return api_fail(SV_ERR_INVALID_ARG, "sv_kernel_time: out is NULL");
  if (reps == 0 || reps > kMaxReps) return api_fail(SV_ERR_INVALID_ARG, "sv_kernel_time: reps must be in [1, 2^20]");
  if (flush_bytes > kMaxFlush) return api_fail(SV_ERR_INVALID_ARG, "sv_kernel_time: flush_bytes exceeds 2^34");
  PerfState *ps = perf_state(k->device);
  std::lock_guard<std::mutex> lock(ps->mu);
  hipError_t e;
  while (ps->events.size() < 2 * (size_t)reps) {
    hipEvent_t ev = nullptr;
    e = hipEventCreate(&ev);
    if (e != hipSuccess) return api_hip_fail(e, "hipEventCreate");
    ps->events.push_back(ev);
  }
  const uint64_t flush_vec = flush_bytes / sizeof(uint4);
  if (flush_vec && ps->flush_cap < flush_vec * sizeof(uint4)) {
    if (ps->flush) (void)hipFree(ps->flush);
    ps->flush = nullptr;
    ps->flush_cap = 0;
    e = hipMalloc((void **)&ps->flush, flush_vec * sizeof(uint4));
    if (e != hipSuccess) {
      ps->flush = nullptr;
      return api_fail(SV_ERR_ALLOC, "sv_kernel_time: cannot allocate the flush buffer");
    }
    ps->flush_cap = flush_vec * sizeof(uint4);
  }
  int cus = 0;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, k->device);
  if (e != hipSuccess) return api_hip_fail(e, "hipDeviceGetAttribute");
  const unsigned fill_blocks = (unsigned)std::max<uint64_t>(
      1, std::min<uint64_t>((flush_vec + kBlock - 1) / kBlock, (uint64_t)std::max(cus, 1) * 8));
  hipStream_t st = api_stream();
  for (uint32_t w = 0; w < warmup; ++w) {
    e = launch_once(k, launch, st);
    if (e != hipSuccess) return api_hip_fail(e, "candidate launch (warm-up)");
  }
  for (uint32_t r = 0; r < reps; ++r) {
    if (flush_vec) {
      hipLaunchKernelGGL(fill_kernel, dim3(fill_blocks), dim3(kBlock), 0, st, ps->flush, flush_vec);
      e = hipGetLastError();
      if (e != hipSuccess) return api_hip_fail(e, "flush launch");
    }
    e = hipEventRecord(ps->events[2 * r], st);
    if (e == hipSuccess) e = launch_once(k, launch, st);
    if (e == hipSuccess) e = hipEventRecord(ps->events[2 * r + 1], st);
    if (e != hipSuccess) return api_hip_fail(e, "timed candidate launch");
  }
  e = hipEventSynchronize(ps->events[2 * (size_t)reps - 1]);
  if (e != hipSuccess) return api_hip_fail(e, "waiting for the timed runs");
  std::vector<double> t(reps);
  double sum = 0.0;
  for (uint32_t r = 0; r < reps; ++r) {
    float ms = 0.0f;
    e = hipEventElapsedTime(&ms, ps->events[2 * r], ps->events[2 * r + 1]);
    if (e != hipSuccess) return api_hip_fail(e, "hipEventElapsedTime");
    t[r] = ms;
    sum += ms;
    if (rep_ms) rep_ms[r] = ms;
  }
  std::sort(t.begin(), t.end());
  out->reps = reps;
  out->reserved = 0;
  out->mean_ms = sum / reps;
  out->median_ms = reps % 2 ? t[reps / 2] : 0.5 * (t[reps / 2 - 1] + t[reps / 2]);
  out->min_ms = t.front();
  out->max_ms = t.back();
  out->perf = 1.0 / out->mean_ms;
  return SV_OK;
}

double sv_reward(int32_t compiled, int32_t valid, double perf) {
  const double c = compiled ? 1.0 : 0.0;
  if (!(compiled && valid)) return -1.0 + c;   // the performance term is absent unless C and V hold
  if (!(perf >= 0.0)) return std::numeric_limits<double>::quiet_NaN();
  return -1.0 + c + c * 1.0 * perf;
}

}  // extern "C"

// sv_files.hip -- test data as files (sv_synth_file, sv_compare_file): the
// scaffold of the paper's generated programs reads its inputs from binary
// files and writes its outputs to binary files (Sec. 4.1), so synthesized
// inputs go straight into files and candidate outputs are checked from files,
// each read with its declared element type.
//
// Both are pipelines over 64 MiB chunks.  Synthesis: chunk k is generated on
// the device (sv_synth_window) and copied to pinned host memory while the host
// writes chunk k - 1 to the file.  Check: one reader thread per file fills a
// ring of pinned buffers while the device checks the chunk before;
// chunk reports are merged exactly (counts summed, first index offset by the
// chunk start, maxima taken, fp64 error sums added in chunk order).
#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <cmath>
#include <condition_variable>
#include <cstring>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "sv_internal.h"

namespace sv {
namespace {

constexpr uint64_t kChunkBytes = 64ull << 20;   // a multiple of 16 bytes and of every Philox block's span
constexpr int kRing = 3;                       // pinned buffers per file in the check's read-ahead ring

size_t item_size(int32_t dtype) { return item_bytes(dtype); }

int io_fail(const char *what, const char *path) {
  const std::string msg = std::string(what) + " '" + path + "': " + std::strerror(errno);
  return api_fail(SV_ERR_IO, msg.c_str());
}

// Staging of the file pipelines, per device, allocated on first use and kept
// (pinning hundreds of MiB costs tens of milliseconds per call otherwise):
// kRing pinned chunks per file side and two device chunks.  One file call per
// device at a time.
struct Staging {
  std::mutex mu;
  void *host[2][kRing] = {};
  void *dev[2] = {};
};

std::mutex g_staging_mu;
std::vector<Staging *> g_staging;

int staging(Staging **out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return api_hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> g(g_staging_mu);
  if ((size_t)dev >= g_staging.size()) g_staging.resize(dev + 1, nullptr);
  if (!g_staging[dev]) g_staging[dev] = new Staging;
  *out = g_staging[dev];
  return SV_OK;
}

// Allocates what is still missing (called with st->mu held).
int fill_staging(Staging *st) {
  for (int side = 0; side < 2; ++side) {
    for (int k = 0; k < kRing; ++k) {
      if (st->host[side][k]) continue;
      if (hipHostMalloc(&st->host[side][k], kChunkBytes, hipHostMallocDefault) != hipSuccess) {
        st->host[side][k] = nullptr;
        return api_fail(SV_ERR_ALLOC, "pinned staging buffer");
      }
    }
    if (!st->dev[side] && hipMalloc(&st->dev[side], kChunkBytes) != hipSuccess) {
      st->dev[side] = nullptr;
      return api_fail(SV_ERR_ALLOC, "device staging buffer");
    }
  }
  return SV_OK;
}

struct Fd {
  int fd = -1;
  ~Fd() {
    if (fd >= 0) (void)::close(fd);
  }
};

bool write_all(int fd, const void *p, size_t bytes) {
  const char *c = (const char *)p;
  while (bytes) {
    const ssize_t w = ::write(fd, c, bytes);
    if (w < 0 && errno == EINTR) continue;
    if (w <= 0) return false;
    c += w;
    bytes -= (size_t)w;
  }
  return true;
}

bool read_all(int fd, void *p, size_t bytes, uint64_t offset) {
  char *c = (char *)p;
  while (bytes) {
    const ssize_t r = ::pread(fd, c, bytes, (off_t)offset);
    if (r < 0 && errno == EINTR) continue;
    if (r <= 0) return false;
    c += r;
    bytes -= (size_t)r;
    offset += (uint64_t)r;
  }
  return true;
}

void merge_report(sv_report &acc, const sv_report &r, uint64_t offset) {
  acc.n += r.n;
  acc.mismatches += r.mismatches;
  if (acc.first_mismatch < 0 && r.first_mismatch >= 0) acc.first_mismatch = (int64_t)offset + r.first_mismatch;
  acc.max_abs_err = std::fmax(acc.max_abs_err, r.max_abs_err);
  acc.max_rel_err = std::fmax(acc.max_rel_err, r.max_rel_err);
  acc.err_sum += r.err_sum;
  acc.nan_ref += r.nan_ref;
  acc.nan_cand += r.nan_cand;
  acc.inf_ref += r.inf_ref;
  acc.inf_cand += r.inf_cand;
}

}  // namespace

void files_shutdown() {
  std::lock_guard<std::mutex> g(g_staging_mu);
  for (Staging *st : g_staging) {
    if (!st) continue;
    std::lock_guard<std::mutex> lock(st->mu);
    for (int side = 0; side < 2; ++side) {
      for (int k = 0; k < kRing; ++k) {
        if (st->host[side][k]) (void)hipHostFree(st->host[side][k]);
        st->host[side][k] = nullptr;
      }
      if (st->dev[side]) (void)hipFree(st->dev[side]);
      st->dev[side] = nullptr;
    }
  }
}

}  // namespace sv

using namespace sv;

extern "C" {

int sv_synth_file(const char *path, uint64_t seed, uint64_t stream_id, int32_t dtype, int32_t dist,
                  const sv_dist_params *params, uint64_t n) {
  api_clear_error();
  if (!path) return api_fail(SV_ERR_INVALID_ARG, "sv_synth_file: path is NULL");
  // validate everything a window synthesis would, before touching the file
  int rc = sv_synth_window(seed, stream_id, dtype, dist, params, 0, 0, nullptr);
  if (rc) return rc;
  if (n > (1ull << 60)) return api_fail(SV_ERR_INVALID_ARG, "sv_synth_file: n exceeds 2^60");
  const size_t isz = item_size(dtype);
  const uint64_t chunk = kChunkBytes / isz;    // elements; a multiple of every distribution's block size
  Fd f;
  f.fd = ::open(path, O_WRONLY | O_CREAT | O_TRUNC | O_CLOEXEC, 0644);
  if (f.fd < 0) return io_fail("sv_synth_file: cannot create", path);
  if (n == 0) return SV_OK;
  Staging *stg;
  if ((rc = staging(&stg))) return rc;
  std::lock_guard<std::mutex> lock(stg->mu);
  if ((rc = fill_staging(stg))) return rc;
  void *dev[2] = {stg->dev[0], stg->dev[1]}, *host[2] = {stg->host[0][0], stg->host[1][0]};
  hipEvent_t done[2] = {nullptr, nullptr};
  for (int k = 0; k < 2; ++k) {
    hipError_t e = hipEventCreateWithFlags(&done[k], hipEventDisableTiming);
    if (e != hipSuccess) {
      for (int j = 0; j < k; ++j) (void)hipEventDestroy(done[j]);
      return api_hip_fail(e, "hipEventCreate");
    }
  }
  struct EventGuard {
    hipEvent_t *e;
    ~EventGuard() {
      (void)hipEventDestroy(e[0]);
      (void)hipEventDestroy(e[1]);
    }
  } guard{done};
  hipStream_t st = api_stream();
  const uint64_t nchunks = (n + chunk - 1) / chunk;
  for (uint64_t k = 0; k <= nchunks; ++k) {
    if (k < nchunks) {                          // generate chunk k and start its copy to the host
      const uint64_t off = k * chunk, m = std::min(chunk, n - off);
      rc = sv_synth_window(seed, stream_id, dtype, dist, params, off, m, dev[k % 2]);
      if (rc) return rc;
      hipError_t e = hipMemcpyAsync(host[k % 2], dev[k % 2], m * isz, hipMemcpyDeviceToHost, st);
      if (e == hipSuccess) e = hipEventRecord(done[k % 2], st);
      if (e != hipSuccess) return api_hip_fail(e, "sv_synth_file: copy to host");
    }
    if (k > 0) {                                // meanwhile write chunk k - 1
      const uint64_t j = k - 1, off = j * chunk, m = std::min(chunk, n - off);
      hipError_t e = hipEventSynchronize(done[j % 2]);
      if (e != hipSuccess) return api_hip_fail(e, "sv_synth_file: waiting for a chunk");
      if (!write_all(f.fd, host[j % 2], m * isz)) return io_fail("sv_synth_file: cannot write", path);
    }
  }
  if (::close(f.fd) != 0) {
    f.fd = -1;
    return io_fail("sv_synth_file: cannot close", path);
  }
  f.fd = -1;
  return SV_OK;
}

int sv_compare_file(const char *ref_path, const char *cand_path, uint64_t n, int32_t dtype, double rtol,
                    double atol, int32_t equal_nan, sv_report *report) {
  api_clear_error();
  if (!ref_path || !cand_path || !report) return api_fail(SV_ERR_INVALID_ARG, "sv_compare_file: NULL argument");
  // validate dtype and tolerances exactly as sv_compare does, with no device work
  int rc = sv_compare(nullptr, nullptr, 0, dtype, rtol, atol, equal_nan, report);
  if (rc) return rc;
  if (n > (1ull << 60)) return api_fail(SV_ERR_INVALID_ARG, "sv_compare_file: n exceeds 2^60");
  const size_t isz = item_size(dtype);
  Fd fr, fc;
  fr.fd = ::open(ref_path, O_RDONLY | O_CLOEXEC);
  if (fr.fd < 0) return io_fail("sv_compare_file: cannot open", ref_path);
  fc.fd = ::open(cand_path, O_RDONLY | O_CLOEXEC);
  if (fc.fd < 0) return io_fail("sv_compare_file: cannot open", cand_path);
  for (int which = 0; which < 2; ++which) {
    struct stat sb;
    const int fd = which ? fc.fd : fr.fd;
    const char *path = which ? cand_path : ref_path;
    if (::fstat(fd, &sb) != 0) return io_fail("sv_compare_file: cannot stat", path);
    if ((uint64_t)sb.st_size != n * isz) {
      const std::string msg = std::string("sv_compare_file: '") + path + "' holds " + std::to_string(sb.st_size) +
                              " bytes, not " + std::to_string(n) + " elements of " + std::to_string(isz) + " bytes";
      return api_fail(SV_ERR_INVALID_ARG, msg.c_str());
    }
  }
  sv_report acc;
  std::memset(&acc, 0, sizeof acc);
  acc.first_mismatch = -1;
  if (n == 0) {
    *report = acc;
    return SV_OK;
  }
  const uint64_t chunk = kChunkBytes / isz;
  const uint64_t nchunks = (n + chunk - 1) / chunk;
  Staging *stg;
  if ((rc = staging(&stg))) return rc;
  std::lock_guard<std::mutex> lock(stg->mu);
  if ((rc = fill_staging(stg))) return rc;
  void *dref = stg->dev[0], *dcand = stg->dev[1];

  // one reader thread per file: side s fills ring slot k % kRing with chunk k
  // once the check has released that slot
  std::mutex mu;
  std::condition_variable cv;
  uint64_t filled[2] = {0, 0}, released = 0;
  bool io_error = false, stop = false;
  std::string io_path;
  int io_errno = 0;
  const int fds[2] = {fr.fd, fc.fd};
  const char *paths[2] = {ref_path, cand_path};
  auto read_ahead = [&](int side) {
    for (uint64_t k = 0; k < nchunks; ++k) {
      {
        std::unique_lock<std::mutex> l(mu);
        cv.wait(l, [&] { return stop || k < released + kRing; });
        if (stop) return;
      }
      const uint64_t off = k * chunk, m = std::min(chunk, n - off);
      const bool ok = read_all(fds[side], stg->host[side][k % kRing], m * isz, off * isz);
      const int err = errno;
      std::lock_guard<std::mutex> l(mu);
      if (!ok) {
        if (!io_error) {
          io_error = true;
          io_errno = err;
          io_path = paths[side];
        }
        cv.notify_all();
        return;
      }
      filled[side] = k + 1;
      cv.notify_all();
    }
  };
  std::thread readers[2];
  auto finish = [&](int code) {
    {
      std::lock_guard<std::mutex> l(mu);
      stop = true;
    }
    cv.notify_all();
    for (auto &t : readers)
      if (t.joinable()) t.join();
    return code;
  };
  try {
    readers[0] = std::thread(read_ahead, 0);
    readers[1] = std::thread(read_ahead, 1);
  } catch (...) {
    return finish(api_fail(SV_ERR_ALLOC, "sv_compare_file: cannot start the reader threads"));
  }
  hipStream_t st = api_stream();
  for (uint64_t k = 0; k < nchunks; ++k) {
    {
      std::unique_lock<std::mutex> l(mu);
      cv.wait(l, [&] { return io_error || (filled[0] > k && filled[1] > k); });
      if (io_error) {
        errno = io_errno;
        const std::string p = io_path;
        l.unlock();
        return finish(io_fail("sv_compare_file: cannot read", p.c_str()));
      }
    }
    const uint64_t off = k * chunk, m = std::min(chunk, n - off);
    hipError_t e = hipMemcpyAsync(dref, stg->host[0][k % kRing], m * isz, hipMemcpyHostToDevice, st);
    if (e == hipSuccess) e = hipMemcpyAsync(dcand, stg->host[1][k % kRing], m * isz, hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return finish(api_hip_fail(e, "sv_compare_file: copy to device"));
    sv_report r;
    rc = sv_compare(dref, dcand, m, dtype, rtol, atol, equal_nan, &r);   // returns once the copies are consumed
    if (rc) return finish(rc);
    merge_report(acc, r, off);
    {
      std::lock_guard<std::mutex> l(mu);
      released = k + 1;
    }
    cv.notify_all();
  }
  finish(SV_OK);
  *report = acc;
  return SV_OK;
}

}  // extern "C"

// sv_internal.h -- structures shared by the host entry points and the kernels
// of libsynthverify.  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sv.h"

namespace sv {

// Launch shape (compile-time tunables, defaults chosen by measurement on MI355X).
#ifndef SV_CMP_UNROLL
#define SV_CMP_UNROLL 4              // 16-byte units per thread in flight in the check
#endif
#ifndef SV_CMP_STOP_UNROLL
#define SV_CMP_STOP_UNROLL 2         // ... in a stop-at-first check: smaller tiles, less read past a mismatch
#endif
#ifndef SV_CMP_BLOCK
#define SV_CMP_BLOCK 512             // threads per check workgroup
#endif
#ifndef SV_CMP_BLOCKS_PER_CU
#define SV_CMP_BLOCKS_PER_CU 8       // check workgroups per CU, single tensor
#endif
#ifndef SV_CMP_FUSE_UNITS
#define SV_CMP_FUSE_UNITS 4096       // a single tensor of at most this many 16-byte units: one workgroup, no finalize
#endif
#ifndef SV_CMP_LAST_BLOCK_MAX
#define SV_CMP_LAST_BLOCK_MAX 64     // single-tensor grids up to this size: the last workgroup reports, no finalize
#endif
#ifndef SV_CMP_SINGLE_LDS
#define SV_CMP_SINGLE_LDS 61440      // dynamic LDS bytes per single-tensor check workgroup, unused: two such
#endif                               // workgroups share a CU's 160 KB, not three (measured faster)
#ifndef SV_CMP_BATCH_BLOCKS_PER_CU
#define SV_CMP_BATCH_BLOCKS_PER_CU 16   // check workgroups per CU, batched
#endif
#ifndef SV_CMP_STOP_BLOCKS_PER_CU
#define SV_CMP_STOP_BLOCKS_PER_CU 12    // ... batched, stop at first mismatch
#endif
#ifndef SV_SYNTH_BLOCKS_PER_CU
#define SV_SYNTH_BLOCKS_PER_CU 64    // synthesis workgroups per CU
#endif
#ifndef SV_SYNTH_NT_BYTES
#define SV_SYNTH_NT_BYTES (1ull << 30)   // single-tensor outputs of at least this many bytes: non-temporal stores
#endif

constexpr int kBlock = 256;          // threads per workgroup of every streaming kernel
constexpr int kCmpBlock = SV_CMP_BLOCK;   // threads per workgroup of the check kernel
#ifndef SV_SYNTH_TILE_ROUNDS
#define SV_SYNTH_TILE_ROUNDS 32      // at most this many vectors per thread in a tile of the batched synthesis
#endif
#ifndef SV_SYNTH_TILES_PER_CU
#define SV_SYNTH_TILES_PER_CU 32     // ... as long as a batch still has this many tiles per CU
#endif
constexpr int kWave = 64;            // CDNA wavefront
constexpr uint64_t kNone = ~0ull;    // "no mismatch yet"

// ----------------------------------------------------------------- synthesis
struct SynthParams {
  uint32_t k0, k1, s0, s1;      // Philox key (seed) and substream words
  float a, span;                // uniform: a + span * U
  float mean, std;              // normal and the normal part of SPECIAL
  int64_t lo;                   // integer range
  uint64_t range;               // hi - lo + 1 (0 stands for 2^64: the whole int64 range)
  uint32_t half;                // permutation: bits of each Feistel half
  uint32_t gate;                // special: an element is a candidate when its gate byte is below this
  uint64_t t_nan, t_inf, t_den, t_zero;   // special: cumulative class thresholds on a candidate's class word
  double a64, span64;           // fp64 uniform: a + span U53
  uint64_t e0;                  // tensor index of out[0] (a window of the tensor; 0 for a whole tensor)
  uint64_t c0;                  // e0 / E, the first Philox block (used when E divides e0)
};

hipError_t launch_synth(int32_t dtype, int32_t dist, const SynthParams &p, uint64_t n, void *out,
                        int cus, hipStream_t stream);

hipError_t launch_eval_transform(int32_t which, const uint32_t *in, uint64_t n, uint32_t *out, int cus,
                                 hipStream_t stream);

// One job of a batched synthesis (device table).  Output vector u of a job
// (16 bytes, V elements) covers elements [u V, u V + V); tiles of kBlock
// vectors are laid end to end over the jobs.
struct SynthJob {
  SynthParams p;
  void *out;
  uint64_t n;
  uint64_t nvec;                // ceil(n / V)
  uint64_t tile_begin;          // first tile of this job
  int32_t kind;                 // dist * 4 + dtype
  int32_t vec_ok;               // out is 16-byte aligned
};

// Vectors per thread in a tile of a batch of total_vecs 16-byte vectors.
inline uint32_t synth_tile_rounds(uint64_t total_vecs, int cus) {
  const uint64_t r = total_vecs / ((uint64_t)cus * SV_SYNTH_TILES_PER_CU * kBlock);
  return (uint32_t)(r < 1 ? 1 : r > SV_SYNTH_TILE_ROUNDS ? SV_SYNTH_TILE_ROUNDS : r);
}
hipError_t launch_synth_batched(const SynthJob *jobs, uint32_t njobs, uint64_t total_tiles, uint32_t rounds,
                                int cus, hipStream_t stream);

// ----------------------------------------------------------------- candidates
struct PerturbParams {
  uint32_t k0, k1, s0, s1;
  uint64_t threshold;           // selected iff w0 < threshold (floor(p 2^32))
  float value;                  // ADD_AT delta, SCALE half-width
  uint32_t bits;                // SET_AT pattern
  int32_t op;
};

hipError_t launch_perturb_elementwise(int32_t dtype, const PerturbParams &p, uint64_t n,
                                      const void *ref, void *cand, int cus, hipStream_t stream);
hipError_t launch_perturb_indexed(int32_t dtype, const PerturbParams &p, const uint64_t *idx_dev,
                                  uint64_t nidx, const void *ref, void *cand, hipStream_t stream);

// ----------------------------------------------------------------- checking
// A "unit" is 16 bytes of one segment: 4 fp32 / int32 or 8 bf16 elements.
// Segments are laid end to end in unit space; workgroup b owns the units
// [b * chunk, (b + 1) * chunk) of that space and writes one partial per
// segment piece it touches, into slot b + s (distinct for every (b, s) pair
// that occurs, because both b and s grow along the unit space).
//
// Stop-at-first launches lay the workgroups out by segment instead: segment s
// gets stop_blocks(units, chunk) workgroups of its own, from workgroup w0 on,
// which sweep it together from the front, workgroup i taking tiles i, i + g,
// i + 2g, ... (a tile is kStopTile = kCmpBlock * SV_CMP_STOP_UNROLL units, one
// iteration of a workgroup); each writes one partial, into slot b.  A mismatch found in a tile
// is posted to the segment's word in `firsts`, so that the segment's other
// workgroups, which are all near that tile, stop there too.
struct SegDesc {
  const void *ref;
  const void *cand;
  uint64_t n;
  uint64_t unit_begin;          // first unit of this segment in the batch's unit space
  double rtol, atol;
  int32_t dtype;
  int32_t equal_nan;
  int32_t vec_ok;               // both pointers 16-byte aligned
  uint32_t w0, w1;              // the first and last check workgroup holding units of it (for a
                                // stop-at-first launch its own workgroups, w0 .. w1 in slots w0 ..;
                                // otherwise slot b + s of workgroup b), so the finalize divides nothing
};

constexpr uint64_t kCmpTile = (uint64_t)kCmpBlock * SV_CMP_UNROLL;   // units per workgroup iteration
constexpr uint64_t kStopTile = (uint64_t)kCmpBlock * SV_CMP_STOP_UNROLL;   // ... of a stop-at-first launch
constexpr uint64_t kMaxStopBlocks = 0xFFFFFFFFull / kCmpBlock;   // a grid's work-items fit in 32 bits
constexpr size_t kFirstStride = 16;   // uint64 words between the segments' words in `firsts` (128 bytes)

// Workgroups of one segment in a stop-at-first launch: a share of about
// `chunk` units each, and no more workgroups than tiles.
__host__ __device__ inline uint64_t stop_blocks(uint64_t units, uint64_t chunk) {
  const uint64_t by_chunk = (units + chunk - 1) / chunk, tiles = (units + kStopTile - 1) / kStopTile;
  return by_chunk < tiles ? by_chunk : tiles;
}

struct Partial {
  uint64_t mism;
  uint64_t first;               // kNone if no mismatch
  double maxabs, maxrel, sum;
  uint64_t nan_r, nan_c, inf_r, inf_c;
};

// What the finalize of a check needs: its segments, the layout of its
// partials, where its reports and completion word go.  The finalize kernel
// runs one workgroup per segment on it; a check whose finalize was left to
// the next check launched on its stream is finished by that launch's first
// workgroups instead (the same code, the same bits).
struct FinalizeArgs {
  const SegDesc *segs;          // device table (batched) or nullptr (single: `single`)
  SegDesc single;
  uint32_t nseg;                // workgroups of the finalize (1 for a single tensor)
  uint64_t chunk;               // units per check workgroup
  const Partial *partials;
  uint32_t *counter;            // arrivals of its workgroups, zero between launches
  int32_t stop_at_first;
  sv_report *reports;
  uint64_t *done;
  uint64_t seq;
};

struct CompareArgs {
  const SegDesc *segs;          // device table (batched) or nullptr (single)
  SegDesc single;               // the segment of a single-tensor check
  uint32_t nseg;
  uint64_t total_units;
  uint64_t chunk;               // units per workgroup
  Partial *partials;            // nblocks + nseg slots
  uint32_t *counter;            // finalize arrivals, zero between launches
  int32_t stop_at_first;        // batched: each failing segment checked only up to its first mismatch
  uint64_t *firsts;             // stop-at-first: word s * kFirstStride of segment s holds
                                // (uint32 seq) << 32 | (2^32 - 1 - t), t the first tile found
                                // with a mismatch in this launch (larger is earlier)
  int32_t fused;                // one tensor, no finalize: 1 = the only workgroup reports, 2 = the last one does
  sv_report *reports;           // nseg reports, in host-mapped pinned memory
  uint64_t *done;               // host-mapped word that receives `seq` once every report is written
  uint64_t seq;
  uint32_t nprev;               // > 0: workgroups 0 .. nprev - 1 finish an earlier check first
  FinalizeArgs prev;
};

// ----------------------------------------------------------------- host helpers
// Shared by the entry-point files; defined in sv_api.hip.
hipStream_t api_stream();                         // the calling thread's stream
void api_clear_error();
int api_fail(int code, const char *msg);          // records msg, returns code
int api_hip_fail(hipError_t e, const char *what);
void perf_shutdown();                             // sv_perf.hip: frees its per-device state
void files_shutdown();                            // sv_files.hip: frees its staging buffers

__host__ __device__ inline uint32_t item_bytes(int32_t dtype) {
  switch (dtype) {
    case SV_BF16: case SV_F16: return 2;
    case SV_F64: case SV_I64: return 8;
    case SV_U8: return 1;
    default: return 4;
  }
}

__host__ __device__ inline uint64_t units_of(int32_t dtype, uint64_t n) {
  const uint64_t per = 16 / item_bytes(dtype);
  return (n + per - 1) / per;
}

// The check kernel (dtype_mask: OR of (1 << dtype) over the segments with
// elements), and the finalize kernel that turns its partials into reports.
hipError_t launch_compare(const CompareArgs &args, uint32_t nblocks, uint32_t dtype_mask, hipStream_t stream);
hipError_t launch_finalize(const FinalizeArgs &f, hipStream_t stream);
FinalizeArgs finalize_args(const CompareArgs &args);
hipError_t launch_fill_u64(uint64_t *p, uint64_t n, uint64_t value, hipStream_t stream);

}  // namespace sv

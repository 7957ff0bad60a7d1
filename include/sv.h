/*
 * sv.h -- C ABI of libsynthverify: seeded synthesis of test inputs and the
 * elementwise functional check of candidate-kernel outputs, on one AMD
 * Instinct MI355X (gfx950).
 *
 * The operations are the data-parallel core of Synthesis-Based Verification
 * in "CUDA-Harness" (arXiv 2609.00058), Sec. 4.2:
 *   - sv_synth produces isolated, reproducible test data (Sec. 4.2.1: test
 *     inputs are synthesized apart from kernel generation, from a broad numeric
 *     range); sv_synth_window any slice of such a tensor, sv_synth_batched
 *     many tensors in one launch;
 *   - sv_compare evaluates the functional validation rule, Eq. (1),
 *       V(K, x, y) = I[ |K(x) - y| <= atol + rtol * |y| ],
 *     element by element, y being the reference output and K(x) the candidate;
 *   - sv_compare_batched checks many outputs in one launch, one report each,
 *     for the progressive, fail-fast validation of Sec. 4.2.2
 *     (sv_compare_batched_mode: each failing output only up to its first
 *     mismatch); sv_compare_submit / sv_compare_batched_submit and
 *     sv_compare_wait run the same checks without waiting for the reports;
 *   - sv_kernel_load / sv_kernel_launch / sv_kernel_time / sv_kernel_free and
 *     sv_reward: the performance stage and the reward (Eq. 3 and 4);
 *   - sv_synth_file and sv_compare_file: test data as raw binary files, the
 *     way the generated programs of Sec. 4.1 exchange it.
 * sv_perturb derives candidates from a reference (test workloads),
 * sv_eval_transform evaluates the building blocks of the normal transform
 * (diagnostics), sv_profile_* times the library's own kernels.
 *
 * Conventions.  All functions return an sv_status (0 on success).  On error
 * nothing is launched and sv_last_error() returns a message for the calling
 * thread.  No C++ exception crosses this interface.  Device pointers are
 * caller-owned HIP device memory on the current device; the library never
 * frees them.  Host pointers are read or written only during the call.
 * Work is issued on the stream set by sv_set_stream() for the calling thread
 * (the null stream by default).  The library owns a per-device scratch area
 * (partial reductions, segment table, report staging) that it allocates on
 * first use, grows when needed and releases in sv_shutdown(); calls that use
 * it on the same device are serialised by a lock, and checks of one device
 * run in submission order.
 *
 * One HIP runtime per process.  The library links libamdhip64.so.7 by that
 * name.  A process that also uses another copy of the runtime (PyTorch ships
 * its own) must load that copy first, so that the library binds to it: with
 * the library loaded first, the process ends up with two runtimes, and the
 * library's sees no device (every call fails with SV_ERR_HIP).  The Python
 * binding imports torch before it loads the library.
 */
#ifndef SV_H
#define SV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SV_ABI_VERSION 1

enum {
  SV_OK = 0,
  SV_ERR_INVALID_ARG = -1, /* null pointer with n > 0, bad tolerance or parameter, size overflow */
  SV_ERR_UNSUPPORTED = -2, /* unknown dtype / dist / op, or an unsupported combination          */
  SV_ERR_HIP = -3,         /* a HIP runtime call failed; the message carries hipGetErrorString  */
  SV_ERR_ALLOC = -4,       /* scratch allocation failed                                         */
  SV_ERR_IO = -5           /* a file could not be opened, read or written (sv_*_file)           */
};

/* Element types.  Storage is contiguous, little-endian, 1-D.  fp16 is IEEE
 * binary16, bf16 the upper half of an fp32. */
enum { SV_F32 = 0, SV_BF16 = 1, SV_I32 = 2, SV_F16 = 3, SV_F64 = 4, SV_U8 = 5, SV_I64 = 6 };

/* Distributions of sv_synth. */
enum {
  SV_UNIFORM = 0,   /* [a, b): fp32, bf16, fp16, fp64                                */
  SV_NORMAL = 1,    /* N(mean, std^2) by Box-Muller: fp32, bf16, fp16, fp64          */
  SV_INT_RANGE = 2, /* integers uniform on [lo, hi] inclusive: int32, uint8, int64   */
  SV_SPECIAL = 3,   /* NaN / +-Inf / denormal / +-0 mix, else N(mean, std^2): fp32, bf16, fp16, fp64 */
  SV_PERMUTATION = 4 /* the values lo .. hi, each once, in a seeded order: int32, uint8, int64 */
};

typedef struct {
  double a, b;                            /* SV_UNIFORM                             */
  double mean, std;                       /* SV_NORMAL and the normal part of SPECIAL */
  int64_t lo, hi;                         /* SV_INT_RANGE, SV_PERMUTATION; within the output type */
  double p_nan, p_inf, p_denorm, p_zero;  /* SV_SPECIAL class probabilities, sum <= 1 */
} sv_dist_params;

/* Result of the check of one tensor (or one segment of a batch). */
typedef struct {
  uint64_t n;              /* elements checked                                        */
  uint64_t mismatches;     /* elements failing Eq. (1)                                */
  int64_t first_mismatch;  /* smallest failing index, -1 if none                      */
  double max_abs_err;      /* max |K(x) - y| over pairs where both are finite, else 0 */
  double max_rel_err;      /* max |K(x) - y| / |y| over those pairs (0/0 -> 0, d/0 -> +Inf) */
  double err_sum;          /* fp64 sum of |K(x) - y| over those pairs                 */
  uint64_t nan_ref, nan_cand, inf_ref, inf_cand;  /* NaN / Inf counts on each side    */
} sv_report;

/* One tensor pair of a batched check. */
typedef struct {
  const void *ref;    /* device: reference output y                    */
  const void *cand;   /* device: candidate output K(x), same dtype and n */
  uint64_t n;         /* elements; 0 allowed                           */
  int32_t dtype;      /* any SV_ element type                           */
  double rtol, atol;  /* finite, >= 0; ignored (and not checked) for the integer types */
  int32_t equal_nan;  /* nonzero: NaN vs NaN agrees                     */
} sv_segment;

/*
 * sv_synth -- fill out[0..n) with element i of the seeded sequence.
 *
 * Element i is a function of (seed, stream_id, i) only: Philox4x32-10
 * (Salmon et al., SC'11) keyed by the seed, with counter (block index,
 * stream_id), where block = i / E and E = 4 (uniform, normal, special, uint8
 * range), 8 (bf16 uniform) or 2 (int32 / int64 range).  Uniform: a + (b - a) *
 * (top 24 bits) * 2^-24 in fp32; a bf16 element takes a 16-bit half-word
 * (the low half first), U = h * 2^-16.  Normal: Box-Muller with ln, sin, cos
 * evaluated as fixed fp32 operation sequences (sin and cos from a table of
 * 256 angles), so the bits are reproducible on any IEEE-754 machine.
 * Integer range: lo + floor(R * (hi - lo + 1) / 2^64), R a 64-bit word.
 * Special: the normal sequence with some elements replaced.  Element 4c + k
 * is a candidate when the low byte of word k of normal block c is below
 * S = ceil(256 * (p_nan + p_inf + p_denorm + p_zero)); a candidate takes its
 * class from x = word k of block 2^62 + c against the cumulative thresholds
 * min(floor(p * 2^40 / S), 2^32) (NaN, Inf, denormal, zero; at or above the
 * last it keeps its normal value), and its sign and payload from
 * x * 0x9E3779B9 mod 2^32 (quiet NaN with that payload, Inf, denormal, zero).
 * bf16
 * and fp16 outputs are the round-to-nearest-even of the fp32 value (an fp16
 * NaN keeps its sign and the top 10 fraction bits, bit 0 set if they are all
 * 0).  fp64 outputs: uniform from 53 random bits, U = (R >> 11) 2^-53 with R
 * a 64-bit word (E = 2), a + (b - a) U in fp64; normal and special are the
 * fp32 values widened exactly (a NaN's fraction moved to the top).  int64
 * ranges use the integer-range rule; for the whole int64 range (hi - lo + 1
 * = 2^64) the value is lo + R.  uint8 ranges take one 32-bit word w per
 * element (E = 4): lo + floor(w * (hi - lo + 1) / 2^32).  Permutation:
 * element i = lo + pi(i), pi a bijection of [0, N), N = hi - lo + 1 <= 2^60:
 * a ten-round Feistel network plus a keyed rotation on the smallest
 * even-bit word domain >= N, repeated until the word falls below N, its keys
 * the words of Philox blocks 0 .. 2; n <= N (n < N: a sample without
 * replacement), and a window must lie inside [0, N).  Any slice of a tensor
 * can be regenerated alone.
 *
 * seed, stream_id : generator key and substream (stream_id is not a HIP stream).
 * dtype, dist     : see the enums; other pairs return SV_ERR_UNSUPPORTED.
 * params          : host pointer, read during the call.
 * n, out          : element count and device output (any alignment of the
 *                   element type; 16-byte aligned outputs take the fast path).
 * Asynchronous: returns after the launch.
 */
int sv_synth(uint64_t seed, uint64_t stream_id, int32_t dtype, int32_t dist,
             const sv_dist_params *params, uint64_t n, void *out);

/* One tensor of a batched synthesis: the arguments of one sv_synth call. */
typedef struct {
  uint64_t seed, stream_id;
  int32_t dtype, dist;
  sv_dist_params params;
  uint64_t n;
  void *out;            /* device; outputs of one batch must not overlap */
} sv_synth_job;

/*
 * sv_synth_batched -- njobs sv_synth calls in one launch.
 *
 * Job k writes exactly what sv_synth(jobs[k].seed, jobs[k].stream_id,
 * jobs[k].dtype, jobs[k].dist, &jobs[k].params, jobs[k].n, jobs[k].out)
 * writes.  The work is cut into tiles of 256 to 8,192 16-byte output vectors
 * (larger tiles for larger batches, so that every CU still gets dozens) spread
 * over the whole grid, so many small tensors cost one launch.  jobs is a host
 * array read during the call; its device copy goes through the library's
 * scratch on the calling thread's stream.  Asynchronous: returns after the
 * launch.  Any invalid job fails the whole call before anything is launched.
 */
int sv_synth_batched(const sv_synth_job *jobs, uint32_t njobs);

/*
 * sv_synth_window -- elements [offset, offset + n) of the tensor that
 * sv_synth(seed, stream_id, dtype, dist, params, N, .) produces for any
 * N >= offset + n, written to out[0 .. n): the same bits as that slice (the
 * counter-based generator needs no state from the elements before it), so a
 * tensor can be produced in pieces, on several devices or straight into a file.
 * Arguments and errors as sv_synth; INVALID_ARG if offset + n > 2^60.
 * Asynchronous.
 */
int sv_synth_window(uint64_t seed, uint64_t stream_id, int32_t dtype, int32_t dist, const sv_dist_params *params,
                    uint64_t offset, uint64_t n, void *out);

/*
 * sv_compare -- evaluate Eq. (1) on every element and reduce into *report.
 *
 * Both values are widened exactly to fp64.  If either is NaN the pair agrees
 * only when equal_nan is set and both are NaN; otherwise if either is
 * infinite the pair agrees only when the values are equal; otherwise it
 * agrees when |K(x) - y| <= atol + rtol * |y|, each operation rounded to
 * nearest in fp64 (no fused multiply-add).  Integer pairs (int32, uint8,
 * int64) agree only when equal; tolerances do not apply to them, and an int64
 * difference is formed exactly before it is rounded to fp64 for the report.
 * V(K, x, y) = 1 exactly when report->mismatches == 0.
 *
 * ref, cand : device pointers to n elements of dtype (any element alignment).
 * report    : host pointer, written on success.
 * Synchronous: returns after the report has reached the host.
 */
int sv_compare(const void *ref, const void *cand, uint64_t n, int32_t dtype,
               double rtol, double atol, int32_t equal_nan, sv_report *report);

/*
 * sv_compare_noalloc -- sv_compare for callers that cannot allocate memory
 * (code under HIP graph capture that prepares its work beforehand, tight
 * serving loops, harnesses that forbid hipMalloc): the same check, the same
 * kernels and the same report bits as sv_compare, but its scratch (workgroup
 * partials, arrival counter, report staging) is a fixed array of 295,168
 * bytes in device memory that the library holds on each GPU it runs on until
 * the process ends.  The call allocates nothing: no hipMalloc, hipFree or
 * pinned host memory, on its first call or any other.
 *
 * ref, cand : device pointers to n elements of dtype (any element alignment);
 *             n is limited only as for sv_compare (at most 2^60).
 * report    : host pointer, written on success.
 * Synchronous: the report is copied to the host and the stream synchronised
 * before the call returns.  Calls on one device share its array and are
 * serialised by a lock; two calls that overlapped on one GPU would race on
 * it, which the lock and the synchronous return rule out within a process.
 * Errors as sv_compare, plus UNSUPPORTED when the device's check grid would
 * need more than the 4,095 workgroup partials the array holds (a GPU of more
 * than 511 compute units) or the device index is 64 or more.
 */
int sv_compare_noalloc(const void *ref, const void *cand, uint64_t n, int32_t dtype,
                       double rtol, double atol, int32_t equal_nan, sv_report *report);

/*
 * sv_compare_batched -- sv_compare on nseg independent segments in one launch.
 *
 * Each segment carries its own dtype, tolerances and equal_nan; indices in
 * its report are local to the segment; zero-length segments are allowed and
 * segments may alias.  Work is balanced by bytes across the whole batch.
 * segs, reports : host arrays of nseg entries.  Synchronous.
 */
int sv_compare_batched(const sv_segment *segs, uint32_t nseg, sv_report *reports);

/*
 * sv_compare_batched_mode -- sv_compare_batched with a choice of how far to
 * check a failing output, for the fail-fast validation of Sec. 4.2.2 (where a
 * failing output ends its candidate's validation, e.g. G candidates x their
 * outputs of one round in one call).
 *   mode = SV_CHECK_FULL (0): exactly sv_compare_batched.
 *   mode = SV_CHECK_STOP_AT_FIRST (1): the check of a segment stops near
 *     where it first meets a mismatch (the segment is swept from the front by
 *     workgroups of its own, which tell each other of the mismatches they
 *     find), but every element before the segment's first mismatch is still
 *     checked.  A passing segment gets its full report (its fp64 error sum
 *     may differ from mode 0's in the last bits: another summation order).
 *     A failing one gets n, mismatches = 1 (meaning "at least one") and the
 *     exact first_mismatch; its other fields are 0.
 * Errors as sv_compare_batched; UNSUPPORTED for another mode.
 */
enum { SV_CHECK_FULL = 0, SV_CHECK_STOP_AT_FIRST = 1 };
int sv_compare_batched_mode(const sv_segment *segs, uint32_t nseg, int32_t mode, sv_report *reports);

/*
 * sv_compare_submit, sv_compare_batched_submit, sv_compare_ready,
 * sv_compare_wait -- the checks above without waiting for their reports, so
 * that the next piece of work (the next candidate's launch, the next
 * synthesis, the next check) is already queued while a report travels to the
 * host.  The generation loop of Sec. 4.3 checks G candidates per round, round
 * after round, and the GPU need not idle between them.
 *
 * A submit call validates its arguments exactly as its synchronous
 * counterpart, queues the same kernels on the selected stream and returns at
 * once with *ticket set.  The tensors must stay valid and unchanged until the
 * check has run (work queued later on the same stream runs after it), and the
 * stream must outlive the wait.  sv_compare_wait(ticket, reports, nreports)
 * blocks until that check's reports are on the host and copies them into
 * reports[0..nreports): nreports must be 1 for sv_compare_submit and nseg for
 * a batch (otherwise INVALID_ARG, and the ticket stays pending).  On success,
 * or on a HIP error, the ticket is used up; waiting twice is INVALID_ARG.
 * sv_compare_ready sets *ready to 1 once a wait would not block, else 0.
 *
 * The last step of a submitted single-tensor check (reducing its workgroups'
 * partial results into the report) is left to the next check queued on the
 * same stream, which does it in one of its own workgroups: one kernel launch
 * less per check when checks follow each other.  If no such check comes,
 * sv_compare_wait and sv_compare_ready queue that step themselves (on the
 * check's stream), as does any call that must drain the pending checks, so a
 * report may not be ready after a mere stream synchronization: poll with
 * sv_compare_ready or wait.  The reports are the same bits either way.
 *
 * At most SV_MAX_PENDING_CHECKS submitted checks per device are pending (not
 * yet waited for); one more submit returns INVALID_ARG.  A ticket names its
 * device, so it may be waited for with any device current.  Checks of one
 * device run one after another in submission order, also across streams: a
 * check queued on another stream than the previous check first waits, on
 * the host, until the pending checks have run.  The synchronous calls are a
 * submit and a wait in one, in a slot of their own.
 */
#define SV_MAX_PENDING_CHECKS 16
int sv_compare_submit(const void *ref, const void *cand, uint64_t n, int32_t dtype, double rtol, double atol,
                      int32_t equal_nan, uint64_t *ticket);
int sv_compare_batched_submit(const sv_segment *segs, uint32_t nseg, int32_t mode, uint64_t *ticket);
int sv_compare_ready(uint64_t ticket, int32_t *ready);
int sv_compare_wait(uint64_t ticket, sv_report *reports, uint32_t nreports);

/* Candidate derivation steps of sv_perturb (workload support, not part of the check). */
enum {
  SV_OP_COPY = 0,         /* cand[i] = ref[i]                                              */
  SV_OP_ULP = 1,          /* selected: next value up or down (fp32, bf16)                   */
  SV_OP_SCALE = 2,        /* selected: fmt(fp32(y * fp32(1 + u))), u in [-value, value)     */
  SV_OP_SPECIAL_FLIP = 3, /* selected zeros change sign, selected NaNs change payload       */
  SV_OP_ADD_AT = 4,       /* cand[idx] = fmt(fp32(y) + fp32(value))        (fp32, bf16)     */
  SV_OP_SET_AT = 5,       /* cand[idx] = bits (low 16 bits for bf16)                       */
  SV_OP_FAULT_AT = 6      /* cand[idx] = fmt(y + (1 + |y|)); int32: y + 1 (wrapping)        */
};

typedef struct {
  int32_t op;
  double p;             /* selection probability of ops 1..3, in [0, 1]           */
  double value;         /* ADD_AT delta; SCALE half-width; a finite fp32 value    */
  uint32_t bits;        /* SET_AT pattern                                         */
  const uint64_t *idx;  /* host: element indices of ops 4..6, each < n            */
  uint64_t nidx;
} sv_perturb_plan;

/*
 * sv_perturb -- derive a candidate from a reference (test-workload support).
 *
 * Ops 0..3 write every cand[i] from ref[i]; element i is selected when the
 * first word of Philox(seed, stream_id, block i) is below floor(p * 2^32), the
 * top bit of the second word gives the ulp direction (1 = up) and the NaN
 * payload mask, the top 24 bits of the third word give u.  Ops 4..6 write only
 * the listed elements, from ref.  ref may equal cand.  Synchronous for ops
 * 4..6 (the index list is staged through the scratch area), asynchronous
 * otherwise.
 */
int sv_perturb(uint64_t seed, uint64_t stream_id, int32_t dtype, const sv_perturb_plan *plan,
               uint64_t n, const void *ref, void *cand);

/*
 * sv_eval_transform -- diagnostics: evaluate one building block of the normal
 * transform of sv_synth on caller-given 24-bit inputs, so that it can be
 * compared exhaustively with an independent implementation.
 *   which = SV_EVAL_LN     : out[i] = bits of ln(u1),        u1 = ((in[i] & 0xFFFFFF) + 1) 2^-24
 *   which = SV_EVAL_RADIUS : out[i] = bits of sqrt(-2 ln u1)  (the Box-Muller radius)
 *   which = SV_EVAL_SIN    : out[i] = bits of sin(2 pi (in[i] & 0xFFFFFF) 2^-24)
 *   which = SV_EVAL_COS    : out[i] = bits of cos(2 pi (in[i] & 0xFFFFFF) 2^-24)
 *   which = SV_EVAL_F16    : out[i] = the fp16 bits sv_synth stores for the fp32 bits in[i]
 *   which = SV_EVAL_BF16   : out[i] = the bf16 bits of the hardware conversion sv_synth
 *                            uses for uniform and normal bf16 values (for in[i] not a NaN)
 * in, out: device arrays of n uint32.  Asynchronous.
 */
enum { SV_EVAL_LN = 0, SV_EVAL_RADIUS = 1, SV_EVAL_SIN = 2, SV_EVAL_COS = 3, SV_EVAL_F16 = 4, SV_EVAL_BF16 = 5 };
int sv_eval_transform(int32_t which, const uint32_t *in, uint64_t n, uint32_t *out);

/*
 * ---- Test data as files (Sec. 4.1: the generated program reads its inputs
 * from binary files and writes its outputs to binary files) ----
 *
 * sv_synth_file -- writes the n elements sv_synth would produce to `path`
 * (created or truncated) as raw little-endian values of `dtype`, n * itemsize
 * bytes, nothing else.  Generated on the current device in 64 MiB chunks, the
 * copy of each to the host overlapping the file write of the one before.
 * Synchronous.  Errors: as sv_synth for the distribution arguments; IO when
 * the file cannot be created or written (a partial file may remain); ALLOC.
 *
 * sv_compare_file -- the check of sv_compare between two files that each hold
 * exactly n raw little-endian values of `dtype` (read as that type: an int32
 * file is compared as integers, never reinterpreted as fp32).  Read in 64 MiB
 * chunks by a reader thread ahead of the device; the chunk reports are merged
 * exactly except for err_sum, which adds the chunks' sums in order (within
 * 1e-12 relative of a one-launch check).  Synchronous.  Errors: as sv_compare
 * for dtype and tolerances; IO when a file cannot be opened or read;
 * INVALID_ARG when a file's size is not n * itemsize.
 */
int sv_synth_file(const char *path, uint64_t seed, uint64_t stream_id, int32_t dtype, int32_t dist,
                  const sv_dist_params *params, uint64_t n);
int sv_compare_file(const char *ref_path, const char *cand_path, uint64_t n, int32_t dtype, double rtol,
                    double atol, int32_t equal_nan, sv_report *report);

/*
 * ---- Performance stage and reward (Sec. 4.2.2, Eq. (3); Sec. 4.3, Eq. (4)) ----
 *
 * After a candidate kernel compiles (C of Eq. (2)) and passes the functional
 * check (V, sv_compare), its runtime performance is measured as
 * P_latency = 1 / Latency (Eq. (3)), the latency being the mean over repeated
 * runs (Sec. 5.1), and the three stages combine into the reward
 * r = -1 + C + C V P (Eq. (4)).
 *
 * sv_kernel_load -- load a candidate: a gfx950 code object (an .hsaco image in
 * host memory, `size` bytes, as produced by `hipcc --genco`) and the name of a
 * kernel in it.  On success *out owns the module; release it with
 * sv_kernel_free.  The kernel belongs to the device current at load time.
 * Errors: INVALID_ARG for NULL arguments or size 0; HIP for a code object the
 * runtime rejects or a name it does not contain.
 */
typedef struct sv_kernel sv_kernel;
int sv_kernel_load(const void *code_object, uint64_t size, const char *name, sv_kernel **out);
int sv_kernel_free(sv_kernel *k);

/*
 * One launch of a candidate: grid (in workgroups) and workgroup dimensions,
 * dynamic LDS bytes, and the kernel's arguments packed into one buffer as the
 * kernel's parameter list lays them out (each parameter at its natural
 * alignment).  `args` is host memory read during the call.
 */
typedef struct {
  uint32_t grid[3];
  uint32_t block[3];
  uint32_t shared_bytes;
  uint32_t reserved;            /* 0 */
  const void *args;
  uint64_t args_size;
} sv_launch;

/* Launches the candidate once on the calling thread's stream (asynchronous). */
int sv_kernel_launch(const sv_kernel *k, const sv_launch *launch);

typedef struct {
  uint32_t reps;
  uint32_t reserved;
  double mean_ms;               /* Latency of Eq. (3): mean of the timed runs */
  double median_ms, min_ms, max_ms;
  double perf;                  /* P = 1 / mean_ms, in 1/ms */
} sv_timing;

/*
 * sv_kernel_time -- the performance stage: `warmup` untimed launches, then
 * `reps` launches each bracketed by HIP events on the calling thread's stream.
 * With flush_bytes > 0, a fill of that many bytes of library scratch runs
 * before every timed launch, outside its events, so each run starts with the
 * L2 and Infinity Cache holding none of the candidate's data (256 MiB or more
 * evicts both on MI355X); at most 2^34 bytes.  Waits for the runs; fills *out
 * and, if rep_ms is not NULL, rep_ms[0..reps) with each run's milliseconds.
 * Errors: INVALID_ARG for NULL k / launch / out, reps == 0 or > 2^20, a zero
 * grid or block dimension, more than 1024 threads per workgroup, args NULL
 * with args_size > 0, a kernel loaded on another device; HIP for launch or
 * event failures (a faulting candidate surfaces here); ALLOC for the flush.
 */
int sv_kernel_time(const sv_kernel *k, const sv_launch *launch, uint32_t warmup, uint32_t reps,
                   uint64_t flush_bytes, float *rep_ms, sv_timing *out);

/*
 * Eq. (4): r = -1 + C + C V P, with C = (compiled != 0), V = (valid != 0) and
 * P >= 0 the performance of Eq. (3) (ignored unless C and V hold).  So a
 * kernel that does not compile gets -1, one that compiles but fails the check
 * 0, and a correct one its performance.  Returns NaN for a NaN or negative P
 * when C and V hold.  Pure host arithmetic.
 */
double sv_reward(int32_t compiled, int32_t valid, double perf);

/* HIP stream (hipStream_t) for the calling thread's later calls; NULL = null stream. */
int sv_set_stream(void *hip_stream);

/* Message of the calling thread's last failed call ("" if none).  Valid until its next call. */
const char *sv_last_error(void);

/*
 * Kernel timing.  While enabled (per process), every kernel launch of the
 * library is bracketed by HIP events on its stream (the markers themselves
 * add a few microseconds between launches).  sv_profile_read() waits for the
 * recorded events of one kind, returns their count and total milliseconds,
 * and forgets them.  Kinds: 0 synthesis, 1 check (the streaming kernel of
 * sv_compare / sv_compare_batched; it includes the reduction of an earlier
 * submitted check that it finishes), 2 candidate derivation, 3 the check's
 * finalize kernel (per-segment reduction and report, when it runs as a
 * kernel of its own).
 */
enum { SV_PROF_SYNTH = 0, SV_PROF_COMPARE = 1, SV_PROF_PERTURB = 2, SV_PROF_FINALIZE = 3 };
int sv_profile_enable(int32_t on);
int sv_profile_read(int32_t kind, uint64_t *count, double *total_ms);

/* Frees the scratch areas of every device, after waiting for the device's
 * work.  Later calls allocate again.  Checks still pending are forgotten:
 * sv_compare_wait on their tickets then fails with SV_ERR_INVALID_ARG. */
int sv_shutdown(void);

/*
 * For tests: sets the sequence number of the last check on the calling
 * thread's current device, so that the next check gets last + 1.  Checks
 * number themselves per device; the stop-at-first mode tags words in device
 * memory with the low 32 bits of that number and clears them when the high
 * bits change, and this lets a test cross that boundary without 2^32 checks.
 * Numbers may be set back and repeat.  Tickets of checks waited for before
 * the call must not be used after it.
 * INVALID_ARG while submitted checks of the device are not yet waited for, or
 * for last >= 2^56 - 2^32 (tickets hold 56 bits of it).
 */
int sv_testing_set_sequence(uint64_t last);

int sv_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* SV_H */

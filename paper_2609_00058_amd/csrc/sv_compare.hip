// sv_compare.hip -- the elementwise check of Eq. (1) fused with the report
// reduction (sv_compare, sv_compare_batched).
//
// Memory plan.  The check reads every reference and candidate byte exactly
// once and writes a few hundred bytes, so it is bound by HBM bandwidth.
// Segments are laid end to end in 16-byte units (4 fp32 / int32 or 8 bf16
// elements); workgroup b owns a contiguous chunk of that unit space, so the
// work is balanced by bytes across ragged batches, and inside a chunk the 256
// threads walk consecutive units (each wave reads 1 KiB per operand per
// dwordx4 load, fully coalesced), four units per thread in flight.  Loads are
// non-temporal: the data is used once.
//
// Per element: both values are widened exactly to fp64, d = |a - y|,
// t = atol + rtol |y| (no fma), match = d <= t for finite pairs, else
// identical infinities agree and NaN agrees with NaN under equal_nan.
// Counts (mismatches, NaN, Inf) and the first mismatching index are
// wave-uniform: each predicate's ballot mask is popcounted on the scalar unit,
// and the first index comes from the lowest set lane of the first nonzero
// mismatch mask a wave sees (a wave visits its units in increasing order).
// The fp64 maxima and the sum stay per lane; the relative error d / |y| is
// divided out only when it can beat the lane's running maximum (the test
// d > fp64(m (1 - 2^-50)) |y| never rejects a ratio whose rounded quotient
// exceeds m), which keeps the fp64 division off the streaming path.
//
// Reduction.  Lanes -> wave by xor shuffles, waves -> workgroup through LDS,
// one partial per (workgroup, segment piece) in scratch, then a finalize
// kernel (one wave per segment) combines a segment's partials in a fixed
// order.  No floating-point atomics: reports are bit-reproducible run to run
// for a given device.
#include "sv_device.h"
#include "sv_internal.h"

namespace sv {

constexpr int kUnroll = 4;             // units per thread in flight
constexpr int kWavesPerBlock = kBlock / kWave;

template <int DT> struct Elem;
template <> struct Elem<SV_F32> { static constexpr int V = 4; };
template <> struct Elem<SV_BF16> { static constexpr int V = 8; };
template <> struct Elem<SV_I32> { static constexpr int V = 4; };

// element j of a 16-byte unit, as raw bits
template <int DT>
__device__ __forceinline__ uint32_t lane_elem(const u32x4 &v, int j) {
  if constexpr (DT == SV_BF16) {
    const uint32_t w = v[j >> 1];
    return (j & 1) ? (w >> 16) : (w & 0xFFFFu);
  } else {
    return v[j];
  }
}

template <int DT>
__device__ __forceinline__ uint32_t load_elem(const void *p, uint64_t i) {
  if constexpr (DT == SV_BF16)
    return ((const uint16_t *)p)[i];
  else
    return ((const uint32_t *)p)[i];
}

struct LaneAcc {
  double maxabs, maxrel, mrc, sum;   // mrc = maxrel (1 - 2^-50), the division filter
};

struct WaveAcc {                      // wave-uniform
  uint64_t mism, first, nan_r, nan_c, inf_r, inf_c;
};

// Checks the V elements of one unit (raw bits in yv / av; element j valid when
// bit j of `valid` is set) and folds them into the accumulators.  Lane l holds
// the unit whose first element is wave_e0 + l V.  Must be reached by every lane
// of the wave that is still iterating (ballots).
template <int DT>
__device__ __forceinline__ void check_unit(const u32x4 &yv, const u32x4 &av, uint32_t valid, uint64_t wave_e0,
                                           double rtol, double atol, bool equal_nan, LaneAcc &L, WaveAcc &W) {
  constexpr int V = Elem<DT>::V;
  uint64_t bad_any = 0;
  uint64_t bad[V];
#pragma unroll
  for (int j = 0; j < V; ++j) {
    const bool ok_j = (valid >> j) & 1u;
    const uint32_t yb = lane_elem<DT>(yv, j), ab = lane_elem<DT>(av, j);
    double Y, A;
    bool nan_y = false, nan_a = false, inf_y = false, inf_a = false;
    if constexpr (DT == SV_I32) {
      Y = (double)(int32_t)yb;
      A = (double)(int32_t)ab;
    } else {
      const float yf = DT == SV_BF16 ? as_f32(yb << 16) : as_f32(yb);
      const float af = DT == SV_BF16 ? as_f32(ab << 16) : as_f32(ab);
      nan_y = __builtin_isnan(yf);
      nan_a = __builtin_isnan(af);
      inf_y = __builtin_isinf(yf);
      inf_a = __builtin_isinf(af);
      Y = (double)yf;
      A = (double)af;
    }
    const double d = fabs(A - Y);
    bool match, finite;
    if constexpr (DT == SV_I32) {
      match = (A == Y);
      finite = true;
    } else {
      const double t = atol + rtol * fabs(Y);
      finite = !(nan_y | nan_a | inf_y | inf_a);
      match = finite ? (d <= t) : ((A == Y) || (equal_nan && nan_y && nan_a));
      W.nan_r += __popcll(__ballot(ok_j && nan_y));
      W.nan_c += __popcll(__ballot(ok_j && nan_a));
      W.inf_r += __popcll(__ballot(ok_j && inf_y));
      W.inf_c += __popcll(__ballot(ok_j && inf_a));
    }
    bad[j] = __ballot(ok_j && !match);
    bad_any |= bad[j];
    if (ok_j && finite) {
      L.sum += d;
      L.maxabs = fmax(L.maxabs, d);
      const double ay = fabs(Y);
      if (d > L.mrc * ay) {             // only then can d / |y| exceed the running maximum
        const double rel = d / ay;       // |y| = 0 < d gives +Inf
        if (rel > L.maxrel) {
          L.maxrel = rel;
          L.mrc = rel * 0x1.ffffffffffff8p-1;   // 1 - 2^-50
        }
      }
    }
  }
  if (bad_any) {                        // wave-uniform
#pragma unroll
    for (int j = 0; j < V; ++j) W.mism += __popcll(bad[j]);
    if (W.first == kNone) {
      // lowest lane with a mismatch, then its lowest element; lanes hold
      // consecutive units, so that is the smallest index this wave has seen
      const uint32_t L0 = __builtin_ctzll(bad_any);
      int jj = V - 1;
#pragma unroll
      for (int j = V - 1; j >= 0; --j)
        if ((bad[j] >> L0) & 1ull) jj = j;
      W.first = wave_e0 + (uint64_t)L0 * V + (uint64_t)jj;
    }
  }
}

__device__ __forceinline__ double shfl_xor_d(double v, int m) { return __shfl_xor(v, m, kWave); }

// Merge partial b into a (commutative, associative except for the sum).
__device__ __forceinline__ void merge(Partial &a, const Partial &b) {
  a.mism += b.mism;
  a.first = a.first < b.first ? a.first : b.first;
  a.maxabs = fmax(a.maxabs, b.maxabs);
  a.maxrel = fmax(a.maxrel, b.maxrel);
  a.sum += b.sum;
  a.nan_r += b.nan_r;
  a.nan_c += b.nan_c;
  a.inf_r += b.inf_r;
  a.inf_c += b.inf_c;
}

__device__ __forceinline__ Partial empty_partial() {
  Partial p;
  p.mism = 0; p.first = kNone; p.maxabs = 0.0; p.maxrel = 0.0; p.sum = 0.0;
  p.nan_r = p.nan_c = p.inf_r = p.inf_c = 0;
  return p;
}

// Units [ulo, uhi) of one segment -> a workgroup partial, valid on thread 0.
template <int DT>
__device__ Partial check_piece(const SegDesc &sd, uint64_t ulo, uint64_t uhi, Partial *lds) {
  constexpr int V = Elem<DT>::V;
  const uint32_t tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const u32x4 *yv4 = (const u32x4 *)sd.ref;
  const u32x4 *av4 = (const u32x4 *)sd.cand;
  const double rtol = sd.rtol, atol = sd.atol;
  const bool eqn = sd.equal_nan != 0;
  const uint64_t n = sd.n;
  const bool vec_ok = sd.vec_ok != 0;
  LaneAcc L{0.0, 0.0, 0.0, 0.0};
  WaveAcc W{0, kNone, 0, 0, 0, 0};
  // wave-uniform loop: the wave's first unit of sub-iteration 0 is below uhi
  for (uint64_t base = ulo + wave * kWave; base < uhi; base += (uint64_t)kBlock * kUnroll) {
    u32x4 yv[kUnroll], av[kUnroll];
    uint32_t valid[kUnroll];
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      const uint64_t u = base + (uint64_t)k * kBlock + lane;
      const uint64_t e0 = u * V;
      valid[k] = 0;
      yv[k] = u32x4{0, 0, 0, 0};
      av[k] = u32x4{0, 0, 0, 0};
      if (u < uhi) {
        if (vec_ok && e0 + V <= n) {
          yv[k] = __builtin_nontemporal_load(yv4 + u);
          av[k] = __builtin_nontemporal_load(av4 + u);
          valid[k] = (1u << V) - 1u;
        } else {
#pragma unroll
          for (int j = 0; j < V; ++j) {
            if (e0 + j < n) {
              const uint32_t yb = load_elem<DT>(sd.ref, e0 + j), ab = load_elem<DT>(sd.cand, e0 + j);
              valid[k] |= 1u << j;
              if constexpr (DT == SV_BF16) {
                yv[k][j >> 1] |= (j & 1) ? (yb << 16) : yb;
                av[k][j >> 1] |= (j & 1) ? (ab << 16) : ab;
              } else {
                yv[k][j] = yb;
                av[k][j] = ab;
              }
            }
          }
        }
      }
    }
#pragma unroll
    for (int k = 0; k < kUnroll; ++k) {
      // element index of lane 0's first element in this sub-iteration (wave-uniform)
      const uint64_t wave_e0 = (base + (uint64_t)k * kBlock) * V;
      check_unit<DT>(yv[k], av[k], valid[k], wave_e0, rtol, atol, eqn, L, W);
    }
  }
  // lanes -> wave
#pragma unroll
  for (int m = kWave / 2; m >= 1; m >>= 1) {
    L.sum += shfl_xor_d(L.sum, m);
    L.maxabs = fmax(L.maxabs, shfl_xor_d(L.maxabs, m));
    L.maxrel = fmax(L.maxrel, shfl_xor_d(L.maxrel, m));
  }
  if (lane == 0) {
    Partial p;
    p.mism = W.mism; p.first = W.first;
    p.maxabs = L.maxabs; p.maxrel = L.maxrel; p.sum = L.sum;
    p.nan_r = W.nan_r; p.nan_c = W.nan_c; p.inf_r = W.inf_r; p.inf_c = W.inf_c;
    lds[wave] = p;
  }
  __syncthreads();
  Partial out = lds[0];
  if (tid == 0) {
#pragma unroll
    for (int w = 1; w < kWavesPerBlock; ++w) merge(out, lds[w]);
  }
  __syncthreads();   // lds is reused by the next piece
  return out;
}

// Segment holding unit `u`: the last segment whose first unit is <= u (empty
// segments share their successor's start and are skipped by this rule).
__device__ __forceinline__ uint32_t find_segment(const SegDesc *segs, uint32_t nseg, uint64_t u) {
  uint32_t lo = 0, hi = nseg;          // answer in [lo, hi)
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) / 2;
    if (segs[mid].unit_begin <= u) lo = mid; else hi = mid;
  }
  return lo;
}

template <bool kSingle>
__global__ __launch_bounds__(kBlock) void compare_kernel(CompareArgs args) {
  __shared__ Partial lds[kWavesPerBlock];
  const uint64_t b = blockIdx.x;
  uint64_t lo = b * args.chunk;
  if (lo >= args.total_units) return;
  const uint64_t hi = lo + args.chunk < args.total_units ? lo + args.chunk : args.total_units;
  uint32_t s = kSingle ? 0u : find_segment(args.segs, args.nseg, lo);
  while (lo < hi) {
    const SegDesc sd = kSingle ? args.single : args.segs[s];
    const uint64_t seg_end = sd.unit_begin + units_of(sd.dtype, sd.n);
    const uint64_t piece_hi = hi < seg_end ? hi : seg_end;
    const uint64_t ulo = lo - sd.unit_begin, uhi = piece_hi - sd.unit_begin;
    Partial p;
    if (sd.dtype == SV_F32)
      p = check_piece<SV_F32>(sd, ulo, uhi, lds);
    else if (sd.dtype == SV_BF16)
      p = check_piece<SV_BF16>(sd, ulo, uhi, lds);
    else
      p = check_piece<SV_I32>(sd, ulo, uhi, lds);
    if (threadIdx.x == 0) args.partials[b + s] = p;
    lo = piece_hi;
    if constexpr (!kSingle) {
      ++s;
      while (s < args.nseg && lo < hi && args.segs[s].n == 0) ++s;
    }
  }
}

// One wave per segment: combine the partials of the workgroups that touched
// it, lane l taking slots l, l + 64, ... in order, then a fixed shuffle tree.
template <bool kSingle>
__global__ __launch_bounds__(kWave) void finalize_kernel(CompareArgs args) {
  const uint32_t s = blockIdx.x, lane = threadIdx.x;
  const SegDesc sd = kSingle ? args.single : args.segs[s];
  const uint64_t units = units_of(sd.dtype, sd.n);
  Partial acc = empty_partial();
  if (units) {
    const uint64_t b0 = sd.unit_begin / args.chunk;
    const uint64_t b1 = (sd.unit_begin + units - 1) / args.chunk;
    for (uint64_t b = b0 + lane; b <= b1; b += kWave) merge(acc, args.partials[b + s]);
  }
#pragma unroll
  for (int m = kWave / 2; m >= 1; m >>= 1) {
    Partial o;
    o.mism = __shfl_xor(acc.mism, m, kWave);
    o.first = __shfl_xor(acc.first, m, kWave);
    o.maxabs = shfl_xor_d(acc.maxabs, m);
    o.maxrel = shfl_xor_d(acc.maxrel, m);
    o.sum = shfl_xor_d(acc.sum, m);
    o.nan_r = __shfl_xor(acc.nan_r, m, kWave);
    o.nan_c = __shfl_xor(acc.nan_c, m, kWave);
    o.inf_r = __shfl_xor(acc.inf_r, m, kWave);
    o.inf_c = __shfl_xor(acc.inf_c, m, kWave);
    merge(acc, o);
  }
  if (lane == 0) {
    sv_report r;
    r.n = sd.n;
    r.mismatches = acc.mism;
    r.first_mismatch = acc.first == kNone ? -1 : (int64_t)acc.first;
    r.max_abs_err = acc.maxabs;
    r.max_rel_err = acc.maxrel;
    r.err_sum = acc.sum;
    r.nan_ref = acc.nan_r;
    r.nan_cand = acc.nan_c;
    r.inf_ref = acc.inf_r;
    r.inf_cand = acc.inf_c;
    args.reports[s] = r;
  }
}

hipError_t launch_compare(const CompareArgs &args, uint32_t nblocks, hipStream_t stream, hipEvent_t ev_start,
                          hipEvent_t ev_mid, hipEvent_t ev_stop) {
  const bool single = args.segs == nullptr;
  if (ev_start) (void)hipEventRecord(ev_start, stream);
  if (nblocks) {
    if (single)
      hipLaunchKernelGGL(compare_kernel<true>, dim3(nblocks), dim3(kBlock), 0, stream, args);
    else
      hipLaunchKernelGGL(compare_kernel<false>, dim3(nblocks), dim3(kBlock), 0, stream, args);
  }
  if (ev_mid) (void)hipEventRecord(ev_mid, stream);
  if (single)
    hipLaunchKernelGGL(finalize_kernel<true>, dim3(1), dim3(kWave), 0, stream, args);
  else
    hipLaunchKernelGGL(finalize_kernel<false>, dim3(args.nseg), dim3(kWave), 0, stream, args);
  if (ev_stop) (void)hipEventRecord(ev_stop, stream);
  return hipGetLastError();
}

}  // namespace sv

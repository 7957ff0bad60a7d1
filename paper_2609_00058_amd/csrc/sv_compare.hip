// sv_compare.hip -- the elementwise check of Eq. (1) fused with the report
// reduction (sv_compare, sv_compare_batched).
//
// Memory plan.  The check reads every reference and candidate byte once and
// writes a few hundred bytes, so it is bound by HBM bandwidth.  Segments are
// laid end to end in 16-byte units (16 uint8, 8 bf16 / fp16, 4 fp32 / int32
// or 2 fp64 / int64 elements);
// workgroup b owns a contiguous chunk of that unit space, so work is balanced
// by bytes across ragged batches.  Inside a chunk each wave reads 64
// consecutive units per operand per dwordx4 load (1 KiB, fully coalesced),
// several units per thread in flight; loads are non-temporal because the data
// is used once.
//
// Per element of a floating-point type: both values are widened exactly to
// fp64, d = |a - y|, t = atol + rtol |y| (no fma), and the pair agrees when
// d <= t if both are finite, otherwise when the values are equal (identical
// infinities) or both are NaN under equal_nan.  A wave first checks whether
// every d of its group is finite (true for all but special-value data); then
// it needs one comparison per element and no NaN / Inf classification.
// Integer types agree only when equal and are checked in integer arithmetic
// (check_group_int).  Elements past the end of a segment are loaded as zero
// on both sides, which agrees and adds nothing.
//
// Counts (mismatches, NaN, Inf) and the first mismatching index are
// wave-uniform: predicate ballots popcounted on the scalar unit; the first
// index is the lowest set lane of the first nonzero mismatch ballot a wave
// sees (a wave visits its units in increasing order).  The fp64 maxima and
// the sum stay per lane; d / |y| is divided out only when it can beat the
// lane's running maximum m (the test d > fp64(m (1 - 2^-50)) |y| never
// rejects a quotient that rounds above m while that product is a normal
// number; fp64 inputs also divide where it is not, see may_beat).
//
// Reduction.  Lanes -> wave by DPP moves and xor shuffles, waves ->
// workgroup through LDS, one 72-byte partial per (workgroup, segment piece)
// in scratch slot b + s.  The finalize -- one workgroup per segment, after
// the check -- combines a segment's partials in a fixed order and writes the
// report straight into host-mapped pinned memory, then its last workgroup
// writes the launch's sequence number, which the host spins on.  It runs as
// a kernel of its own behind the check, or, for a submitted check followed
// by another on its stream, in the first workgroups of that next check.  No
// floating-point atomics: reports are bit-reproducible run to run for a
// given device.  A small single tensor needs no finalize: one workgroup, or
// the last of a few dozen, writes the report itself (last_block_report), by
// the same reduction tree.
//
// The partials of a large grid need no device-scope fence inside the check:
// the finalize runs after it.  (On gfx950 such a fence writes back the whole
// L2 of the issuing XCD, which cuts the check to a third of its bandwidth
// when thousands of workgroups each issue one; an in-kernel "last workgroup
// finishes" scheme built from device-scope atomic stores instead of fences
// measured slower than the separate finalize, its chain of round trips to the
// coherence point being longer than a kernel launch.)
#include "sv_device.h"
#include "sv_internal.h"

namespace sv {

constexpr int kUnroll = SV_CMP_UNROLL;   // units per thread in flight
constexpr int kStopUnroll = SV_CMP_STOP_UNROLL;   // ... in a stop-at-first launch (its tile: kStopTile)
constexpr int kWavesPerBlock = kCmpBlock / kWave;

// V elements per 16-byte unit, checked in groups of G.
template <int DT> struct Elem;
template <> struct Elem<SV_F32> { static constexpr int V = 4, G = 4; };
template <> struct Elem<SV_BF16> { static constexpr int V = 8, G = 4; };
template <> struct Elem<SV_I32> { static constexpr int V = 4, G = 4; };
template <> struct Elem<SV_F16> { static constexpr int V = 8, G = 4; };
template <> struct Elem<SV_U8> { static constexpr int V = 16, G = 4; };
template <> struct Elem<SV_F64> { static constexpr int V = 2, G = 2; };
template <> struct Elem<SV_I64> { static constexpr int V = 2, G = 2; };

template <int DT> constexpr bool kIntType = DT == SV_I32 || DT == SV_U8 || DT == SV_I64;
template <int DT> constexpr bool kSmallInt = DT == SV_I32 || DT == SV_U8;   // |a - y| fits 32 bits
template <int DT> constexpr bool kWideType = DT == SV_F64 || DT == SV_I64;   // 64-bit elements

// Element j of a 16-byte unit, for the types up to 32 bits: fp32 bits (bf16
// and fp16 widened exactly) or the integer.
template <int DT>
__device__ __forceinline__ uint32_t elem_bits(const u32x4 &v, int j) {
  if constexpr (DT == SV_BF16)
    return (j & 1) ? (v[j >> 1] & 0xFFFF0000u) : (v[j >> 1] << 16);
  else if constexpr (DT == SV_F16)
    return as_u32(f16_widen((j & 1) ? (v[j >> 1] >> 16) : (v[j >> 1] & 0xFFFFu)));
  else if constexpr (DT == SV_U8)
    return (v[j >> 2] >> (8 * (j & 3))) & 0xFFu;
  else
    return v[j];
}

// Element j of a unit of 64-bit elements.
__device__ __forceinline__ uint64_t elem_bits64(const u32x4 &v, int j) {
  return ((uint64_t)v[2 * j + 1] << 32) | v[2 * j];
}

template <int DT>
__device__ __forceinline__ double widen(uint32_t bits) {
  if constexpr (DT == SV_I32)
    return (double)(int32_t)bits;
  else if constexpr (DT == SV_U8)
    return (double)bits;
  else
    return (double)as_f32(bits);
}

// Operands live in device (global) memory.  A segment's pointers are read
// from the segment table, so the compiler cannot infer their address space
// and would address them as generic (flat) pointers: flat loads also count
// against the LDS / scalar-load counter the loop waits on.  Casting them to
// the global address space gives global loads, as for kernel arguments.
#define kGlobal __attribute__((address_space(1)))

template <int DT>
__device__ __forceinline__ uint64_t load_elem(const void *p, uint64_t i) {
  if constexpr (DT == SV_BF16 || DT == SV_F16)
    return ((const kGlobal uint16_t *)p)[i];
  else if constexpr (DT == SV_U8)
    return ((const kGlobal uint8_t *)p)[i];
  else if constexpr (kWideType<DT>)
    return ((const kGlobal uint64_t *)p)[i];
  else
    return ((const kGlobal uint32_t *)p)[i];
}

// Places element j's raw bits into a unit (the tail of a segment).
template <int DT>
__device__ __forceinline__ void put_elem(u32x4 &v, int j, uint64_t b) {
  if constexpr (DT == SV_BF16 || DT == SV_F16) {
    v[j >> 1] |= (j & 1) ? ((uint32_t)b << 16) : (uint32_t)b;
  } else if constexpr (DT == SV_U8) {
    v[j >> 2] |= (uint32_t)b << (8 * (j & 3));
  } else if constexpr (kWideType<DT>) {
    v[2 * j] = (uint32_t)b;
    v[2 * j + 1] = (uint32_t)(b >> 32);
  } else {
    v[j] = (uint32_t)b;
  }
}

struct LaneAcc {
  double maxabs, maxrel, mrc, sum;   // mrc = maxrel (1 - 2^-50): the division filter
  uint64_t isum;                     // int32 / uint8: exact sum of |a - y| since the last fold into sum
  uint32_t imax;                     // int32 / uint8: max |a - y|
  uint32_t rd, ry;                   // int32 / uint8: max d / |y| as the exact ratio rd / ry (ry = 0: +Inf)
};

struct WaveAcc {                      // wave-uniform
  uint64_t mism, first, nan_r, nan_c, inf_r, inf_c;
};

// Whether d / |y| may round above the running maximum m the lane holds (the
// wave's, as of its last rise): d > fp64(mrc
// |y|) never rejects such a quotient while that product is a normal fp64
// number (its relative rounding error, at most 2^-53, is inside the 2^-50
// margin of mrc).  Widened fp32, bf16 and fp16 values and int64 differences
// keep it normal (m |y| >= 2^-426 once both are nonzero).  fp64 inputs do
// not: below 2^-1022 the product is rounded to a multiple of 2^-1074, an
// absolute error the margin does not cover, and a difference of two finite
// values can overflow to +Inf, whose quotient beats any finite m even where
// the product has overflowed too.  There the quotient is always formed.
template <int DT>
__device__ __forceinline__ bool may_beat(const LaneAcc &L, double d, double ay) {
  const double b = L.mrc * ay;
  if constexpr (DT == SV_F64)
    return d > b || (d > 0.0 && b < 0x1p-1022) || d == __builtin_inf();
  else
    return d > b;
}

// Gives every lane the wave's largest relative error so far (defined with the
// cross-lane steps below).
__device__ __forceinline__ void share_rel(LaneAcc &L);

__device__ __forceinline__ void update_rel(LaneAcc &L, double d, double y) {
  const double rel = d / fabs(y);    // y = 0 < d gives +Inf
  if (rel > L.maxrel) {
    L.maxrel = rel;
    L.mrc = rel * 0x1.ffffffffffff8p-1;   // 1 - 2^-50
  }
}

// Folds elements G g .. G g + G - 1 of one unit (lane l holds the unit whose
// first element is wave_e0 + l V) into the lane accumulators and the wave
// counts; bad[j] receives the ballot of the mismatches of element G g + j.
// Reached by every lane of the wave (ballots).  int64 differences are formed
// exactly and rounded once (fp64 cannot hold every int64); with the zero
// tolerances of integer types the test d <= 0 is then exact equality.
// Pairs holding a NaN or an infinity are decided with wave masks and scalar
// bit operations (kMasks), or with per-lane selects and branches: the
// stop-at-first kernel, whose loop measured faster that way (the candidates
// round's check 285 against 308 us; the single and the batched check faster
// with masks, e.g. 1262 against 1356 us for 2^30 special values).
template <int DT, bool kMasks = true>
__device__ __forceinline__ void check_group(const u32x4 &yv, const u32x4 &av, int g, double rtol, double atol,
                                            bool eqn, LaneAcc &L, WaveAcc &W, uint64_t *bad) {
  constexpr int G = Elem<DT>::G;
  double Y[G], D[G], A[G];
  bool nonfin = false;
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const int e = G * g + j;
    if constexpr (DT == SV_I64) {
      const int64_t yi = (int64_t)elem_bits64(yv, e), ai = (int64_t)elem_bits64(av, e);
      const uint64_t mag = ai >= yi ? (uint64_t)ai - (uint64_t)yi : (uint64_t)yi - (uint64_t)ai;
      Y[j] = (double)yi;
      D[j] = (double)mag;
      A[j] = 0.0;
    } else if constexpr (DT == SV_F64) {
      Y[j] = bits_f64(elem_bits64(yv, e));
      A[j] = bits_f64(elem_bits64(av, e));
      D[j] = fabs(A[j] - Y[j]);
      nonfin |= !__builtin_isfinite(D[j]);
    } else {
      Y[j] = widen<DT>(elem_bits<DT>(yv, e));
      A[j] = 0.0;
      D[j] = fabs(widen<DT>(elem_bits<DT>(av, e)) - Y[j]);
      if constexpr (!kIntType<DT>) nonfin |= !__builtin_isfinite(D[j]);
    }
  }
  bool f[G];
  bool anyf = false;
  if (kIntType<DT> || __ballot(nonfin) == 0) {
    // every pair of this group is finite across the wave
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const double ay = fabs(Y[j]);
      bad[j] = __ballot(!(D[j] <= atol + rtol * ay));
      L.sum += D[j];
      L.maxabs = fmax(L.maxabs, D[j]);
      f[j] = may_beat<DT>(L, D[j], ay);
      anyf |= f[j];
    }
  } else if constexpr (!kMasks) {
#pragma unroll
    for (int j = 0; j < G; ++j) {
      bool ny, na, iy, ia, same;
      if constexpr (DT == SV_F64) {
        ny = __builtin_isnan(Y[j]);
        na = __builtin_isnan(A[j]);
        iy = __builtin_isinf(Y[j]);
        ia = __builtin_isinf(A[j]);
        same = A[j] == Y[j];
      } else {
        const float yf = as_f32(elem_bits<DT>(yv, G * g + j)), af = as_f32(elem_bits<DT>(av, G * g + j));
        ny = __builtin_isnan(yf);
        na = __builtin_isnan(af);
        iy = __builtin_isinf(yf);
        ia = __builtin_isinf(af);
        same = af == yf;
      }
      W.nan_r += __popcll(__ballot(ny));
      W.nan_c += __popcll(__ballot(na));
      W.inf_r += __popcll(__ballot(iy));
      W.inf_c += __popcll(__ballot(ia));
      const bool fin = !(ny | na | iy | ia);
      const double ay = fabs(Y[j]);
      const bool match = fin ? (D[j] <= atol + rtol * ay) : (same || (eqn && ny && na));
      bad[j] = __ballot(!match);
      const double dj = fin ? D[j] : 0.0;
      L.sum += dj;
      L.maxabs = fmax(L.maxabs, dj);
      f[j] = may_beat<DT>(L, dj, ay);
      anyf |= f[j];
    }
  } else {
#pragma unroll
    for (int j = 0; j < G; ++j) {
      // every decision as a wave mask (one ballot per compare), combined
      // with scalar bit operations
      uint64_t ny, na, iy, ia, same;
      bool lane_fin;                     // this lane's pair is finite
      if constexpr (DT == SV_F64) {
        ny = __ballot(__builtin_isnan(Y[j]));
        na = __ballot(__builtin_isnan(A[j]));
        iy = __ballot(__builtin_isinf(Y[j]));
        ia = __ballot(__builtin_isinf(A[j]));
        same = __ballot(A[j] == Y[j]);
        lane_fin = __builtin_isfinite(Y[j]) && __builtin_isfinite(A[j]);   // (their difference may overflow)
      } else {
        // the fp32 values (bf16 and fp16 widened exactly) have the classes,
        // and compare equal exactly when, the fp64 ones do; their difference
        // is finite exactly when both are
        const float yf = as_f32(elem_bits<DT>(yv, G * g + j)), af = as_f32(elem_bits<DT>(av, G * g + j));
        ny = __ballot(__builtin_isnan(yf));
        na = __ballot(__builtin_isnan(af));
        iy = __ballot(__builtin_fabsf(yf) > 0x1.fffffep+127f);
        ia = __ballot(__builtin_fabsf(af) > 0x1.fffffep+127f);
        same = __ballot(af == yf);
        lane_fin = __builtin_fabs(D[j]) <= 0x1.fffffffffffffp+1023;   // a compare the ballot takes as it is
      }
      const uint64_t fin = __ballot(lane_fin);
      W.nan_r += __popcll(ny);
      W.nan_c += __popcll(na);
      W.inf_r += __popcll(iy);
      W.inf_c += __popcll(ia);
      const double ay = fabs(Y[j]);
      const uint64_t within = __ballot(D[j] <= atol + rtol * ay);
      // a pair holding a NaN or an infinity matches when the values are equal
      // (equal infinities) or, with equal_nan, both are NaN
      const uint64_t match = (fin & within) | (~fin & (same | (eqn ? ny & na : 0ull)));
      bad[j] = ~match & __ballot(true);
      const double dj = lane_fin ? D[j] : 0.0;
      L.sum += dj;
      L.maxabs = fmax(L.maxabs, dj);
      f[j] = may_beat<DT>(L, dj, ay);
      anyf |= f[j];
    }
  }
  if (__ballot(anyf)) {              // a lane may have a new relative maximum
#pragma unroll
    for (int j = 0; j < G; ++j)
      if (f[j]) update_rel(L, D[j], Y[j]);
    // the report needs only the largest quotient of all: filtering every lane
    // against the wave's largest divides far less often where most pairs
    // differ (a lane alone sees few pairs, so its own maximum keeps rising)
    share_rel(L);
  }
}

// Elements G g .. G g + G - 1 of a unit of int32 or uint8 elements.  Eq. (1)
// is plain equality for integers, and d = |a - y| < 2^32 is exact in 32
// bits, so the decision, the sum (exact, folded into the fp64 sum once per
// tile), the maximum and the largest d / |y| need no floating point: the
// ratio is kept exactly as rd / ry and compared by cross-multiplication
// (d ry > rd |y|, products below 2^63); starting from 0 / 1, a d > 0 at y = 0
// makes it +Inf (ry = 0), which nothing then beats.  Rounding being
// monotone, the one fp64 division at the end gives the largest of the
// rounded quotients.
template <int DT>
__device__ __forceinline__ void check_group_int(const u32x4 &yv, const u32x4 &av, int g, LaneAcc &L,
                                                uint64_t *bad) {
  constexpr int G = Elem<DT>::G;
  uint32_t gsum = 0;                 // uint8: the group's sum, at most 4 * 255
#pragma unroll
  for (int j = 0; j < G; ++j) {
    const int e = G * g + j;
    uint32_t d, ay;
    bool beats;
    if constexpr (DT == SV_I32) {
      const int32_t yi = (int32_t)yv[e], ai = (int32_t)av[e];
      d = ai >= yi ? (uint32_t)ai - (uint32_t)yi : (uint32_t)yi - (uint32_t)ai;
      ay = yi < 0 ? 0u - (uint32_t)yi : (uint32_t)yi;
      L.isum += d;
      beats = (uint64_t)d * L.ry > (uint64_t)L.rd * ay;
    } else {
      const uint32_t yb = elem_bits<DT>(yv, e), ab = elem_bits<DT>(av, e);
      d = ab >= yb ? ab - yb : yb - ab;
      ay = yb;
      gsum += d;
      beats = d * L.ry > L.rd * ay;  // products below 2^16
    }
    bad[j] = __ballot(d != 0);
    L.imax = d > L.imax ? d : L.imax;
    L.rd = beats ? d : L.rd;
    L.ry = beats ? ay : L.ry;
  }
  if constexpr (DT == SV_U8) L.isum += gsum;
}

// Folds the exact integer sum into the fp64 sum.
__device__ __forceinline__ void fold_int_sum(LaneAcc &L) {
  L.sum += (double)L.isum;
  L.isum = 0;
}

// One unit: its groups, then the mismatch count and, for the first
// mismatching unit a wave sees, the smallest mismatching index.
template <int DT, bool kMasks = true>
__device__ __forceinline__ void check_unit(const u32x4 &yv, const u32x4 &av, uint64_t wave_e0, double rtol,
                                           double atol, bool eqn, LaneAcc &L, WaveAcc &W) {
  constexpr int V = Elem<DT>::V;
  constexpr int G = Elem<DT>::G;
  if constexpr (kIntType<DT>) {
    // every lane's unit bitwise equal: every d is 0 and nothing is counted
    const bool same = yv[0] == av[0] && yv[1] == av[1] && yv[2] == av[2] && yv[3] == av[3];
    if (__ballot(!same) == 0) return;
  }
  uint64_t bad[V];                   // wave masks, kept in scalar registers
#pragma unroll
  for (int g = 0; g < V / G; ++g) {
    if constexpr (kSmallInt<DT>)
      check_group_int<DT>(yv, av, g, L, bad + G * g);
    else
      check_group<DT, kMasks>(yv, av, g, rtol, atol, eqn, L, W, bad + G * g);
  }
  uint64_t any = 0;
#pragma unroll
  for (int j = 0; j < V; ++j) any |= bad[j];
  if (any) {                         // wave-uniform, rare
#pragma unroll
    for (int j = 0; j < V; ++j) W.mism += __popcll(bad[j]);
    if (W.first == kNone) {
      // lowest lane with a mismatch, then its lowest element
      const uint32_t l0 = __builtin_ctzll(any);
      int jj = V - 1;
#pragma unroll
      for (int j = V - 1; j >= 0; --j)
        if ((bad[j] >> l0) & 1ull) jj = j;
      W.first = wave_e0 + (uint64_t)l0 * V + (uint64_t)jj;
    }
  }
}

// ---- cross-lane steps of the wave reductions
// Step k pairs each lane with one holding the other half of its 2^(k+1)-lane
// group: for groups of 2, 4, 8 and 16 lanes through DPP moves inside the VALU
// (quad permutes, then the half-row and row mirrors, whose partner lies in the
// other half of the group, which after the earlier steps holds one uniform
// value), for 32 and 64 lanes through the LDS crossbar.  Every merge is
// commutative, so the result is one fixed tree, identical on every lane.
constexpr int kDppXor1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppMirror = 0x140;

template <int kStep>
__device__ __forceinline__ uint32_t lane_pair32(uint32_t v) {
  if constexpr (kStep == 0) return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kDppXor1, 0xF, 0xF, false);
  else if constexpr (kStep == 1) return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kDppXor2, 0xF, 0xF, false);
  else if constexpr (kStep == 2) return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kDppHalfMirror, 0xF, 0xF, false);
  else if constexpr (kStep == 3) return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kDppMirror, 0xF, 0xF, false);
  else return (uint32_t)__shfl_xor((int)v, kStep == 4 ? 16 : 32, kWave);
}

template <int kStep>
__device__ __forceinline__ uint64_t lane_pair(uint64_t v) {
  return ((uint64_t)lane_pair32<kStep>((uint32_t)(v >> 32)) << 32) | lane_pair32<kStep>((uint32_t)v);
}

template <int kStep>
__device__ __forceinline__ double lane_pair(double v) {
  return __longlong_as_double((long long)lane_pair<kStep>((uint64_t)__double_as_longlong(v)));
}

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

template <int kStep>
__device__ __forceinline__ void merge_step(Partial &acc) {
  Partial o;
  o.mism = lane_pair<kStep>(acc.mism);
  o.first = lane_pair<kStep>(acc.first);
  o.maxabs = lane_pair<kStep>(acc.maxabs);
  o.maxrel = lane_pair<kStep>(acc.maxrel);
  o.sum = lane_pair<kStep>(acc.sum);
  o.nan_r = lane_pair<kStep>(acc.nan_r);
  o.nan_c = lane_pair<kStep>(acc.nan_c);
  o.inf_r = lane_pair<kStep>(acc.inf_r);
  o.inf_c = lane_pair<kStep>(acc.inf_c);
  merge(acc, o);
}

__device__ __forceinline__ void wave_merge(Partial &acc) {
  merge_step<0>(acc);
  merge_step<1>(acc);
  merge_step<2>(acc);
  merge_step<3>(acc);
  merge_step<4>(acc);
  merge_step<5>(acc);
}

__device__ __forceinline__ void share_rel(LaneAcc &L) {
  double m = L.maxrel;
  m = fmax(m, lane_pair<0>(m));
  m = fmax(m, lane_pair<1>(m));
  m = fmax(m, lane_pair<2>(m));
  m = fmax(m, lane_pair<3>(m));
  m = fmax(m, lane_pair<4>(m));
  m = fmax(m, lane_pair<5>(m));
  L.maxrel = m;
  L.mrc = m * 0x1.ffffffffffff8p-1;   // 1 - 2^-50, as in update_rel
}

__device__ __forceinline__ uint64_t dbits(double x) { return (uint64_t)__double_as_longlong(x); }

// ---- hand-off to the host
__device__ __forceinline__ void wait_memory() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// The report as ten 64-bit words, in sv_report's field order.
__device__ __forceinline__ void report_words(const Partial &r, uint64_t n, uint64_t *v) {
  v[0] = n;
  v[1] = r.mism;
  v[2] = r.first == kNone ? ~0ull : r.first;     // -1 as int64 when there is no mismatch
  v[3] = dbits(r.maxabs);
  v[4] = dbits(r.maxrel);
  v[5] = dbits(r.sum);
  v[6] = r.nan_r;
  v[7] = r.nan_c;
  v[8] = r.inf_r;
  v[9] = r.inf_c;
}
constexpr int kReportWords = 10;

// Thread 0's merged result r becomes the report *dst: ten lanes of wave 0
// write its words together, with system-scope stores.  Reached by every
// thread of the workgroup.
__device__ __forceinline__ void publish_report(const Partial &r, uint64_t n, sv_report *dst) {
  __shared__ uint64_t words[kReportWords];
  if (threadIdx.x == 0) report_words(r, n, words);
  __syncthreads();
  if (threadIdx.x < kReportWords)
    __hip_atomic_store((uint64_t *)dst + threadIdx.x, words[threadIdx.x], __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_SYSTEM);
}

// Called by one thread of a check that is its own only workgroup, once its
// report is written: waits for those stores, then hands the sequence number
// to the host.
__device__ __forceinline__ void signal_done(const CompareArgs &args) {
  wait_memory();
  __hip_atomic_store(args.done, args.seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

template <int kStep>
__device__ __forceinline__ void lane_step(LaneAcc &L) {
  L.sum += lane_pair<kStep>(L.sum);
  L.maxabs = fmax(L.maxabs, lane_pair<kStep>(L.maxabs));
  L.maxrel = fmax(L.maxrel, lane_pair<kStep>(L.maxrel));
}

// What a stop-at-first workgroup shares: the segment's word in `firsts` and
// an LDS copy of the smallest tile known to the workgroup to hold a mismatch.
struct StopCtx {
  uint64_t *word;
  uint32_t epoch;               // the launch's tag in the word's high half
  uint32_t *lim;                // LDS
};

// Early exit (kStop): a wave leaves the segment once its next tile t starts
// past its own first mismatch, or lies past a tile that holds one.  Only
// units past a known mismatch are skipped, so the segment's first mismatch
// (the smallest over its waves) stays exact; every other statistic of a
// failing segment is dropped from its report.  A wave posts its own first
// mismatch once: to the workgroup's LDS minimum and, when that improves it,
// to the segment's word (an atomic max of the tagged, inverted tile index; a
// word left by an earlier launch carries another tag and counts as nothing).
// Each iteration a wave reads the LDS minimum; one wave per iteration (each
// wave on its first) also reads the segment's word, which costs one uncached
// 8-byte load per workgroup per tile instead of one per wave.
template <int V>
__device__ __forceinline__ bool leave_segment(const StopCtx &sc, uint64_t t, uint64_t wbase, const WaveAcc &W,
                                              bool &told, uint32_t it, uint32_t wave, uint32_t lane) {
  if (W.first != kNone && !told) {
    told = true;
    const uint32_t f = (uint32_t)(W.first / V / kStopTile);
    if (lane == 0) {
      const uint32_t old = __hip_atomic_fetch_min(sc.lim, f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      if (f < old)
        __hip_atomic_fetch_max(sc.word, ((uint64_t)sc.epoch << 32) | (0xFFFFFFFFu - f), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  if (wbase * V > W.first) return true;
  uint32_t lim = __hip_atomic_load(sc.lim, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  if (it == 0 || it % kWavesPerBlock == wave) {
    const uint64_t w = __hip_atomic_load(sc.word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if ((uint32_t)(w >> 32) == sc.epoch) {
      const uint32_t g = 0xFFFFFFFFu - (uint32_t)w;
      if (g < lim) {
        lim = g;
        if (lane == 0) __hip_atomic_fetch_min(sc.lim, g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    }
  }
  return t / kStopTile > __builtin_amdgcn_readfirstlane(lim);
}

// The tiles ulo, ulo + step, ... below uhi of one segment (units, relative to
// the segment; ulo and step multiples of the tile, kCmpTile units, or
// kStopTile for a stop-at-first launch) -> a workgroup partial, valid on
// thread 0.  A plain launch passes its contiguous piece with step = kCmpTile;
// a stop-at-first launch its share of the segment's tiles.
template <int DT, bool kStop = false, bool kMasks = true>
__device__ Partial check_piece(const SegDesc &sd, uint64_t ulo, uint64_t uhi, uint64_t step, const StopCtx *sc,
                               Partial *lds) {
  constexpr int V = Elem<DT>::V;
  constexpr int kU = kStop ? kStopUnroll : kUnroll;   // units per thread per tile
  const uint32_t tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const kGlobal u32x4 *yv4 = (const kGlobal u32x4 *)sd.ref;
  const kGlobal u32x4 *av4 = (const kGlobal u32x4 *)sd.cand;
  const double rtol = sd.rtol, atol = sd.atol;
  const bool eqn = sd.equal_nan != 0;
  const uint64_t n = sd.n;
  // units below full_end are whole and 16-byte loadable
  const uint64_t full_end = sd.vec_ok ? (uhi < n / V ? uhi : n / V) : 0;
  LaneAcc L{0.0, 0.0, 0.0, 0.0, 0, 0, 0, 1};
  WaveAcc W{0, kNone, 0, 0, 0, 0};
  const uint64_t wofs = (uint64_t)wave * kWave;   // this wave's units in a tile: wofs + k * kCmpBlock + lane
  bool told = false;
  uint32_t it = 0;
  uint64_t t = ulo;
  // whole tiles: kU sub-iterations of kCmpBlock units, every unit full
  for (; t + wofs + (uint64_t)(kU - 1) * kCmpBlock + kWave <= full_end; t += step, ++it) {
    if constexpr (kStop) {
      if (leave_segment<V>(*sc, t, t + wofs, W, told, it, wave, lane)) break;
    }
    const uint64_t base = t + wofs;
    u32x4 yv[kU], av[kU];
#pragma unroll
    for (int k = 0; k < kU; ++k) {
      const uint64_t u = base + (uint64_t)k * kCmpBlock + lane;
      yv[k] = __builtin_nontemporal_load(yv4 + u);
      av[k] = __builtin_nontemporal_load(av4 + u);
    }
#pragma unroll
    for (int k = 0; k < kU; ++k)
      check_unit<DT, kMasks>(yv[k], av[k], (base + (uint64_t)k * kCmpBlock) * V, rtol, atol, eqn, L, W);
    if constexpr (kSmallInt<DT>) fold_int_sum(L);
  }
  // the rest, one sub-iteration at a time, guarded (same unit order); a plain
  // launch's tiles are contiguous, a stop-at-first share jumps by `step`
  // after each tile's last sub-iteration
  for (uint64_t base = t + wofs, k = 0; base < uhi; ++k) {
    if constexpr (kStop) {
      if (k % kU == 0 && leave_segment<V>(*sc, base - wofs, base, W, told, it++, wave, lane)) break;
      if (base * V > W.first) break;
    }
    const uint64_t u = base + lane;
    u32x4 yv = u32x4{0, 0, 0, 0}, av = u32x4{0, 0, 0, 0};
    if (u < full_end) {
      yv = __builtin_nontemporal_load(yv4 + u);
      av = __builtin_nontemporal_load(av4 + u);
    } else if (u < uhi) {
      const uint64_t e0 = u * V;
#pragma unroll
      for (int j = 0; j < V; ++j) {
        if (e0 + j < n) {
          put_elem<DT>(yv, j, load_elem<DT>(sd.ref, e0 + j));
          put_elem<DT>(av, j, load_elem<DT>(sd.cand, e0 + j));
        }
      }
    }
    check_unit<DT, kMasks>(yv, av, base * V, rtol, atol, eqn, L, W);
    if constexpr (kSmallInt<DT>) fold_int_sum(L);
    if constexpr (kStop)
      base += (k % kU == kU - 1) ? step - (uint64_t)(kU - 1) * kCmpBlock : (uint64_t)kCmpBlock;
    else
      base += kCmpBlock;
  }
  if constexpr (kStop) {
    // a mismatch in the wave's last tile: post it for the segment's other workgroups
    if (W.first != kNone && !told && lane == 0) {
      const uint32_t f = (uint32_t)(W.first / V / kStopTile);
      __hip_atomic_fetch_max(sc->word, ((uint64_t)sc->epoch << 32) | (0xFFFFFFFFu - f), __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  if constexpr (kSmallInt<DT>) {
    L.maxabs = (double)L.imax;
    L.maxrel = L.rd == 0 ? 0.0 : (L.ry == 0 ? __builtin_inf() : (double)L.rd / (double)L.ry);
  }
  // lanes -> wave -> workgroup
  lane_step<0>(L);
  lane_step<1>(L);
  lane_step<2>(L);
  lane_step<3>(L);
  lane_step<4>(L);
  lane_step<5>(L);
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
  __syncthreads();   // lds is reused
  return out;
}

// Segment holding unit u: the last segment whose first unit is <= u (empty
// segments share their successor's start and are skipped by this rule).
__device__ __forceinline__ uint32_t find_segment(const SegDesc *segs, uint32_t nseg, uint64_t u) {
  uint32_t lo = 0, hi = nseg;
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) / 2;
    if (segs[mid].unit_begin <= u) lo = mid; else hi = mid;
  }
  return lo;
}

// The reduction of a segment's partials P[b0 .. b1] into its report, by a
// workgroup of kFinBlock threads: thread t merges slots b0 + t, b0 + t +
// kFinBlock, ... in order, then a fixed shuffle tree and the waves in order.
// The result is valid on thread 0.  The finalize kernel runs it with four
// slots in flight per thread; a check kernel that finishes an earlier check
// in its first workgroups runs it with one (kFour = false), which keeps the
// check's registers at what its own loop needs.  The merges are the same in
// either case, and so are the bits.
constexpr int kFinBlock = kCmpBlock;             // finalize threads per segment
constexpr int kFinWaves = kFinBlock / kWave;
static_assert(kFinWaves == kWavesPerBlock, "a check workgroup runs the finalize's tree");

template <bool kFour>
__device__ Partial reduce_partials(const Partial *P, uint64_t b0, uint64_t b1, Partial *lds) {
  const uint32_t tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  Partial acc = empty_partial();
  uint64_t b = b0 + tid;
  if constexpr (!kFour) {
    for (; b <= b1; b += kFinBlock) merge(acc, P[b]);
  } else {
    for (; b + 3 * kFinBlock <= b1; b += 4 * kFinBlock) {
      const Partial p0 = P[b], p1 = P[b + kFinBlock], p2 = P[b + 2 * kFinBlock], p3 = P[b + 3 * kFinBlock];
      merge(acc, p0);
      merge(acc, p1);
      merge(acc, p2);
      merge(acc, p3);
    }
    // at most three left: all loaded before the first merge (one memory round
    // trip instead of up to three), merged in the same order
    const bool h0 = b <= b1, h1 = b + kFinBlock <= b1, h2 = b + 2 * kFinBlock <= b1;
    Partial q0, q1, q2;
    if (h0) q0 = P[b];
    if (h1) q1 = P[b + kFinBlock];
    if (h2) q2 = P[b + 2 * kFinBlock];
    if (h0) merge(acc, q0);
    if (h1) merge(acc, q1);
    if (h2) merge(acc, q2);
  }
  wave_merge(acc);
  if (lane == 0) lds[wave] = acc;
  __syncthreads();
  Partial r = lds[0];
  if (tid == 0) {
#pragma unroll
    for (int w = 1; w < kFinWaves; ++w) merge(r, lds[w]);
  }
  __syncthreads();   // lds is reused
  return r;
}

// Segment s of a finished check: its report, then (one thread) the arrival of
// this workgroup among the nwg that finalize the check; the last to arrive
// clears the counter and hands the sequence number to the host.  Each
// workgroup waits for its own stores before it arrives.  The counter's reset
// need not land before the sequence number: the next launch that uses it
// starts after this one has ended.
template <bool kFour>
__device__ void finalize_segment(const FinalizeArgs &f, uint32_t s, uint32_t nwg, Partial *lds) {
  const SegDesc sd = f.segs ? f.segs[s] : f.single;
  const uint64_t units = units_of(sd.dtype, sd.n);
  if (units != 0) {                  // empty segments are reported by the host
    // the segment's workgroups and their slots: a piece of workgroups b0..b1 in
    // slots b + s, or (stop at first) workgroups of its own in slots b
    const bool own = f.segs && f.stop_at_first;
    const Partial r = reduce_partials<kFour>(f.partials + (own ? 0 : s), sd.w0, sd.w1, lds);
    publish_report(r, sd.n, f.reports + s);
  }
  if (threadIdx.x == 0) {
    wait_memory();
    if (nwg > 1) {
      if (__hip_atomic_fetch_add(f.counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != nwg - 1) return;
      __hip_atomic_store(f.counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __hip_atomic_store(f.done, f.seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

// One workgroup per segment, behind the check kernel; the reports go into
// host-mapped memory.
__global__ __launch_bounds__(kFinBlock) void finalize_kernel(FinalizeArgs f) {
  __shared__ Partial lds[kFinWaves];
  finalize_segment<true>(f, blockIdx.x, gridDim.x, lds);
}

// kMask: the set of dtypes (bit 1 << dtype) the segments of this launch use;
// only their code paths are compiled in, which keeps register pressure at
// what the widest of them needs.
// The check of one piece for the element types in kMask (bit 1 << dtype):
// with one type the code of that type only, else a branch on the segment's.
template <int kMask, bool kStop, bool kMasks, int DT = 0>
__device__ __forceinline__ Partial check_any(const SegDesc &sd, uint64_t ulo, uint64_t uhi, uint64_t step,
                                             const StopCtx *sc, Partial *lds) {
  if constexpr (DT > SV_I64) {
    return empty_partial();                         // not reached: the host passes types in kMask only
  } else if constexpr ((kMask & (1 << DT)) == 0) {
    return check_any<kMask, kStop, kMasks, DT + 1>(sd, ulo, uhi, step, sc, lds);
  } else if constexpr ((kMask >> (DT + 1)) == 0) {
    return check_piece<DT, kStop, kMasks>(sd, ulo, uhi, step, sc, lds);   // the last type in the mask
  } else {
    if (sd.dtype == DT) return check_piece<DT, kStop, kMasks>(sd, ulo, uhi, step, sc, lds);
    return check_any<kMask, kStop, kMasks, DT + 1>(sd, ulo, uhi, step, sc, lds);
  }
}

// A small single-tensor grid (at most one wave's worth of workgroups): the
// last workgroup to finish merges every partial and writes the report, so no
// finalize kernel is launched.  Each workgroup makes its partial visible with
// a device-scope fence before it arrives on the counter; the last one fences
// again before it reads.  (Such a fence writes back the issuing XCD's L2: a
// few dozen of them cost little, thousands are what rule this scheme out for
// large grids.)  Lane t of wave 0 takes partial t and the wave reduces them
// by the finalize kernel's tree, the other lanes and waves holding empty
// partials there, so the report is bit-identical to the finalize's.
static_assert(SV_CMP_LAST_BLOCK_MAX <= kWave, "the last workgroup merges the partials in one wave");

__device__ __forceinline__ void last_block_report(const CompareArgs &args, const Partial &p, uint64_t n) {
  __shared__ uint32_t is_last;
  const uint32_t tid = threadIdx.x;
  if (tid == 0) {
    args.partials[blockIdx.x] = p;
    __threadfence();
    is_last = __hip_atomic_fetch_add(args.counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
              gridDim.x - 1;
  }
  __syncthreads();
  if (!is_last) return;
  __threadfence();
  Partial acc = empty_partial();
  if (tid < kWave) {
    if (tid < gridDim.x) merge(acc, args.partials[tid]);
    wave_merge(acc);
  }
  publish_report(acc, n, args.reports);
  if (tid == 0) {
    __hip_atomic_store(args.counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    wait_memory();
    __hip_atomic_store(args.done, args.seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

// Segment owning workgroup b of a stop-at-first launch: the last one whose
// first workgroup is <= b (segments without units own none and are skipped).
__device__ __forceinline__ uint32_t find_block_segment(const SegDesc *segs, uint32_t nseg, uint32_t b) {
  uint32_t lo = 0, hi = nseg;
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) / 2;
    if (segs[mid].w0 <= b) lo = mid; else hi = mid;
  }
  return lo;
}

template <bool kSingle, int kMask, bool kStop = false>
__global__ __launch_bounds__(kCmpBlock) void compare_kernel(CompareArgs args) {
  __shared__ Partial lds[kWavesPerBlock];
  uint64_t b = blockIdx.x;
  if constexpr (!kStop) {
    if (args.nprev) {
      // the first workgroups finish the earlier check left to this launch (its
      // partials are complete: that check kernel ended before this one began);
      // stop-at-first launches take none: their loop needs the registers
      if (b < args.nprev) {
        finalize_segment<false>(args.prev, (uint32_t)b, args.nprev, lds);
        return;
      }
      b -= args.nprev;
    }
  }
  if constexpr (kStop) {
    // one segment per workgroup: its tiles i, i + g, ... (i = b - w0)
    __shared__ uint32_t lim;
    const uint32_t s = find_block_segment(args.segs, args.nseg, (uint32_t)b);
    const SegDesc sd = args.segs[s];
    const uint64_t units = units_of(sd.dtype, sd.n);
    const uint64_t g = stop_blocks(units, args.chunk);
    if (threadIdx.x == 0) lim = 0xFFFFFFFFu;
    __syncthreads();
    const StopCtx sc{args.firsts + (size_t)s * kFirstStride, (uint32_t)args.seq, &lim};
    const Partial p = check_any<kMask, true, false>(sd, (b - sd.w0) * kStopTile, units, g * kStopTile, &sc, lds);
    if (threadIdx.x == 0) args.partials[b] = p;
  } else {
    uint64_t lo = b * args.chunk;
    const uint64_t hi = lo + args.chunk < args.total_units ? lo + args.chunk : args.total_units;
    uint32_t s = kSingle ? 0u : find_segment(args.segs, args.nseg, lo);
    while (lo < hi) {
      const SegDesc sd = kSingle ? args.single : args.segs[s];
      const uint64_t seg_end = sd.unit_begin + units_of(sd.dtype, sd.n);
      const uint64_t piece_hi = hi < seg_end ? hi : seg_end;
      const uint64_t ulo = lo - sd.unit_begin, uhi = piece_hi - sd.unit_begin;
      const Partial p = check_any<kMask, false, true>(sd, ulo, uhi, kCmpTile, nullptr, lds);
      if constexpr (kSingle) {
        if (args.fused == 1) {         // the only workgroup: its partial is the whole result
          publish_report(p, sd.n, args.reports);
          if (threadIdx.x == 0) signal_done(args);
          return;
        }
        if (args.fused == 2) {
          last_block_report(args, p, sd.n);
          return;
        }
      }
      if (threadIdx.x == 0) args.partials[b + s] = p;
      if constexpr (kSingle) return;   // one segment: the chunk is a single piece
      lo = piece_hi;
      if constexpr (!kSingle) {
        ++s;
        while (s < args.nseg && lo < hi && args.segs[s].n == 0) ++s;
      }
    }
  }
}

template <int kMask>
static void launch_masked(const CompareArgs &args, uint32_t nblocks, hipStream_t stream) {
  if (args.segs == nullptr)
    // a single tensor's check runs two workgroups per CU (16 waves), held there by
    // an LDS request it does not use: 80.8 against 82.5 us for 2 x 256 MiB of fp32,
    // 1432 against 1508 us for 2 x 4 GiB of special values, than three per CU
    hipLaunchKernelGGL((compare_kernel<true, kMask>), dim3(nblocks), dim3(kCmpBlock), SV_CMP_SINGLE_LDS, stream, args);
  else if (args.stop_at_first)
    hipLaunchKernelGGL((compare_kernel<false, kMask, true>), dim3(nblocks), dim3(kCmpBlock), 0, stream, args);
  else
    hipLaunchKernelGGL((compare_kernel<false, kMask>), dim3(nblocks), dim3(kCmpBlock), 0, stream, args);
}

// Kernels exist for each type alone, for the mixes of fp32 / bf16 / int32 the
// batched workloads use, and one for any other mix.
hipError_t launch_compare(const CompareArgs &args, uint32_t nblocks, uint32_t dtype_mask, hipStream_t stream) {
  switch (dtype_mask) {
    case 1 << SV_F32: launch_masked<1 << SV_F32>(args, nblocks, stream); break;
    case 1 << SV_BF16: launch_masked<1 << SV_BF16>(args, nblocks, stream); break;
    case 1 << SV_I32: launch_masked<1 << SV_I32>(args, nblocks, stream); break;
    case 1 << SV_F16: launch_masked<1 << SV_F16>(args, nblocks, stream); break;
    case 1 << SV_F64: launch_masked<1 << SV_F64>(args, nblocks, stream); break;
    case 1 << SV_U8: launch_masked<1 << SV_U8>(args, nblocks, stream); break;
    case 1 << SV_I64: launch_masked<1 << SV_I64>(args, nblocks, stream); break;
    case 3: launch_masked<3>(args, nblocks, stream); break;
    case 5: launch_masked<5>(args, nblocks, stream); break;
    case 6: launch_masked<6>(args, nblocks, stream); break;
    case 7: launch_masked<7>(args, nblocks, stream); break;
    default: launch_masked<0x7F>(args, nblocks, stream); break;
  }
  return hipGetLastError();
}

__global__ void fill_u64_kernel(uint64_t *p, uint64_t n, uint64_t value) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (uint64_t)gridDim.x * blockDim.x)
    p[i] = value;
}

hipError_t launch_fill_u64(uint64_t *p, uint64_t n, uint64_t value, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const uint64_t want = (n + kBlock - 1) / kBlock, blocks = want < 1024 ? want : 1024;
  hipLaunchKernelGGL(fill_u64_kernel, dim3((uint32_t)blocks), dim3(kBlock), 0, stream, p, n, value);
  return hipGetLastError();
}

FinalizeArgs finalize_args(const CompareArgs &args) {
  return FinalizeArgs{args.segs, args.single, args.segs ? args.nseg : 1u, args.chunk, args.partials,
                      args.counter, args.stop_at_first, args.reports, args.done, args.seq};
}

hipError_t launch_finalize(const FinalizeArgs &f, hipStream_t stream) {
  hipLaunchKernelGGL(finalize_kernel, dim3(f.nseg), dim3(kFinBlock), 0, stream, f);
  return hipGetLastError();
}

}  // namespace sv

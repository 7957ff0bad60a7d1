// sv_synth.hip -- seeded synthesis of test inputs (sv_synth).
//
// Element i of a tensor is a pure function of (seed, stream, i), so any
// thread can produce any element and any slice can be regenerated alone.  The
// fast path gives every thread one 16-byte output vector per iteration (4
// fp32 / int32 or 8 bf16 elements), computes the Philox blocks that cover it
// (one for uniform and normal fp32 and for uniform bf16, whose elements take
// 16-bit draws; two for normal bf16 and the integer range; special values
// take the normal blocks plus one class block for each block that holds a
// candidate element) and writes it with one dwordx4 store.
// The grid is a fixed multiple of the CU count with a grid-stride loop; the
// ragged tail (fewer than one vector) is written element by element by the
// first threads of the same launch.  Outputs that are not 16-byte aligned, and
// windows that start inside a Philox block, go through a one-element-per-thread
// kernel.  A window of a tensor (out[0] = element e0) is the same bits as the
// slice of the whole tensor: only the counter base moves.  The path is ALU-bound (Philox is
// 20 32x32->64-bit products and 20 XOR pairs per block, of which the uniform
// substream words leave 18 products and 15 three-input XORs per lane when the
// block indices fit 32 bits; Box-Muller adds a logarithm, a square root and a
// sine / cosine pair per two elements).
#include <type_traits>

#include "sv_device.h"
#include "sv_internal.h"

namespace sv {

template <int DIST> struct DistTraits;

// Kernels that draw normal values (normal and special distributions) fill the
// sine / cosine table of the Box-Muller transform first, every thread of the
// workgroup taking part.
template <int DIST>
__device__ __forceinline__ void prepare_distribution() {
  if constexpr (DIST == SV_NORMAL || DIST == SV_SPECIAL) load_sincos_table();
}
template <> struct DistTraits<SV_UNIFORM> { static constexpr int E = 4; };
template <> struct DistTraits<SV_NORMAL> { static constexpr int E = 4; };
template <> struct DistTraits<SV_INT_RANGE> { static constexpr int E = 2; };
template <> struct DistTraits<SV_SPECIAL> { static constexpr int E = 4; };

// Special values: the normal sequence with some elements replaced.  Element
// 4c + k is a candidate when its gate, the low byte of word k of normal
// block c (bits Box-Muller leaves unused), is below p.gate; a candidate's
// class word is word k of Philox block 2^62 + c (block indices the normal
// values, below 2^58, never reach), its sign and payload bits that word
// times 0x9E3779B9 (Fibonacci hashing).
constexpr uint64_t kSpecialClassBlocks = 1ull << 62;
constexpr uint32_t kPayloadHash = 0x9E3779B9u;

// Candidate `x`-word element: its class (cumulative thresholds NaN, Inf,
// denormal, zero; at or above the last it keeps the normal value v).
__device__ __forceinline__ void special_overlay(const SynthParams &p, uint32_t x, uint32_t &v) {
  if (x < p.t_zero) {
    const uint32_t r = x * kPayloadHash;
    const uint32_t sign = r & 0x80000000u;
    const uint32_t m = r & 0x007FFFFFu;
    v = x < p.t_nan   ? sign | 0x7FC00000u | (r & 0x003FFFFFu)
        : x < p.t_inf ? sign | 0x7F800000u
        : x < p.t_den ? sign | (m ? m : 1u)
                      : sign;
  }
}

// Bit k set: element k of a block whose words are w is a special candidate.
__device__ __forceinline__ uint32_t candidates(const SynthParams &p, const u32x4 &w) {
  return ((w.x & 0xFFu) < p.gate ? 1u : 0u) | ((w.y & 0xFFu) < p.gate ? 2u : 0u) |
         ((w.z & 0xFFu) < p.gate ? 4u : 0u) | ((w.w & 0xFFu) < p.gate ? 8u : 0u);
}

// The special elements among the four values v of normal block `block`,
// whose candidates are the set bits of c.
__device__ __forceinline__ void apply_overlay(const SynthParams &p, uint64_t block, uint32_t c, uint32_t *v) {
  const u32x4 q = philox_block(Key{p.k0, p.k1, p.s0, p.s1}, kSpecialClassBlocks + block);
  if (c & 1u) special_overlay(p, q.x, v[0]);
  if (c & 2u) special_overlay(p, q.y, v[1]);
  if (c & 4u) special_overlay(p, q.z, v[2]);
  if (c & 8u) special_overlay(p, q.w, v[3]);
}

// The E element values (fp32 bits or int32 bits) of Philox block `block`.
template <int DIST>
__device__ __forceinline__ void block_values(const SynthParams &p, uint64_t block, uint32_t *v) {
  const Key key{p.k0, p.k1, p.s0, p.s1};
  const u32x4 w = philox_block(key, block);
  if constexpr (DIST == SV_UNIFORM) {
    v[0] = as_u32(p.a + p.span * unit24(w.x));
    v[1] = as_u32(p.a + p.span * unit24(w.y));
    v[2] = as_u32(p.a + p.span * unit24(w.z));
    v[3] = as_u32(p.a + p.span * unit24(w.w));
  } else if constexpr (DIST == SV_NORMAL) {
    float c0, s0, c1, s1;
    box_muller(w.x, w.y, c0, s0);
    box_muller(w.z, w.w, c1, s1);
    v[0] = as_u32(__builtin_fmaf(p.std, c0, p.mean));   // mean + std z, one rounding
    v[1] = as_u32(__builtin_fmaf(p.std, s0, p.mean));
    v[2] = as_u32(__builtin_fmaf(p.std, c1, p.mean));
    v[3] = as_u32(__builtin_fmaf(p.std, s1, p.mean));
  } else if constexpr (DIST == SV_INT_RANGE) {
    // Lemire's multiply-shift: lo + floor(R * range / 2^64), R a 64-bit word
    const uint64_t r0 = ((uint64_t)w.y << 32) | w.x;
    const uint64_t r1 = ((uint64_t)w.w << 32) | w.z;
    v[0] = (uint32_t)(int32_t)(p.lo + (int64_t)__umul64hi(r0, p.range));
    v[1] = (uint32_t)(int32_t)(p.lo + (int64_t)__umul64hi(r1, p.range));
  } else {
    // the normal values of the block, then the overlay of its candidates
    float c0, s0, c1, s1;
    box_muller(w.x, w.y, c0, s0);
    box_muller(w.z, w.w, c1, s1);
    v[0] = as_u32(__builtin_fmaf(p.std, c0, p.mean));
    v[1] = as_u32(__builtin_fmaf(p.std, s0, p.mean));
    v[2] = as_u32(__builtin_fmaf(p.std, c1, p.mean));
    v[3] = as_u32(__builtin_fmaf(p.std, s1, p.mean));
    const uint32_t c = candidates(p, w);
    if (c) apply_overlay(p, block, c, v);
  }
}

// Elements per Philox block of the 4-byte-value kernels (fp32, bf16, int32
// outputs): bf16 uniform values take a 16-bit half-word each, eight per
// block; the others as DistTraits.
template <int DIST, int DT> struct PerBlock { static constexpr int E = DistTraits<DIST>::E; };
template <> struct PerBlock<SV_UNIFORM, SV_BF16> { static constexpr int E = 8; };
template <> struct PerBlock<SV_INT_RANGE, SV_U8> { static constexpr int E = 4; };

// The E = PerBlock<DIST, DT>::E values (fp32 bits or int32 bits) of Philox
// block `block`.  bf16 uniform: element 2j + h of the block takes half h (low
// first) of word j, U = half 2^-16 (exact), a + span U in fp32.
template <int DIST, int DT>
__device__ __forceinline__ void values_of(const SynthParams &p, uint64_t block, uint32_t *v) {
  if constexpr (DIST == SV_UNIFORM && DT == SV_BF16) {
    const u32x4 w = philox_block(Key{p.k0, p.k1, p.s0, p.s1}, block);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[2 * j] = as_u32(p.a + p.span * ((float)(w[j] & 0xFFFFu) * 0x1p-16f));
      v[2 * j + 1] = as_u32(p.a + p.span * ((float)(w[j] >> 16) * 0x1p-16f));
    }
  } else if constexpr (DIST == SV_INT_RANGE && DT == SV_U8) {
    // uint8: a range of at most 256 values from one 32-bit word per element
    const u32x4 w = philox_block(Key{p.k0, p.k1, p.s0, p.s1}, block);
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = (uint32_t)p.lo + __umulhi(w[k], (uint32_t)p.range);
  } else {
    block_values<DIST>(p, block, v);
  }
}

// One 16-byte output vector.  Outputs much larger than the 256 MB Infinity
// Cache are written with non-temporal stores (p.nt, set per launch): cached
// stores leave the output's last-written part in the caches, and the check
// that reads it next measured 8-12 % slower for it (2^30 fp32:
// 1422 against 1241 us after a normal-value synthesis, 1452 against 1307 us
// after special values); outputs that fit the cache keep cached stores, so
// that the check finds them there (2^26 fp32 pairs: 4702 against 4631 GB/s).
// (A compile-time choice: with a run-time branch the compiler merges the two
// stores into one plain store.)
template <bool kNT>
__device__ __forceinline__ void store_vec(u32x4 *out, uint64_t u, const u32x4 &o) {
  if constexpr (kNT)
    __builtin_nontemporal_store(o, out + u);
  else
    out[u] = o;
}

// Two elements as bf16 in one word.  Uniform and normal values are never
// NaN, so the hardware conversion applies; special values go through
// bf16_rne and its NaN rule.
template <int DIST>
__device__ __forceinline__ uint32_t bf16_pair(uint32_t lo, uint32_t hi) {
  if constexpr (DIST == SV_UNIFORM || DIST == SV_NORMAL)
    return bf16x2_rne_not_nan(lo, hi);
  else
    return bf16_rne(lo) | (bf16_rne(hi) << 16);
}

// The two 16-bit values (first in the low half) of the fp32 values lo, hi in
// a narrow output type: the hardware conversions for values that cannot be
// NaN (the normal values of vectors without candidates), the conversions with
// the NaN rules for the rest.
template <int DT>
__device__ __forceinline__ uint32_t narrow_pair_not_nan(uint32_t lo, uint32_t hi) {
  if constexpr (DT == SV_BF16) {
    return bf16x2_rne_not_nan(lo, hi);
  } else {
    asm("" : "+v"(lo), "+v"(hi));   // keep the fp32 rounding of the values
    return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)as_f32(lo)) |
           ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)as_f32(hi)) << 16);
  }
}
template <int DT>
__device__ __forceinline__ uint32_t narrow_pair(uint32_t lo, uint32_t hi) {
  if constexpr (DT == SV_BF16) return bf16_rne(lo) | (bf16_rne(hi) << 16);
  else return f16_rne(lo) | (f16_rne(hi) << 16);
}

template <int DIST, int DT>
__device__ __forceinline__ void store_elem(void *out, uint64_t i, uint32_t x) {
  if constexpr (DT == SV_BF16)
    ((uint16_t *)out)[i] = (uint16_t)bf16_rne(x);
  else if constexpr (DT == SV_F16)
    ((uint16_t *)out)[i] = (uint16_t)f16_rne(x);
  else if constexpr (DT == SV_U8)
    ((uint8_t *)out)[i] = (uint8_t)x;
  else
    ((uint32_t *)out)[i] = x;
}

// Vectors [0, nvec) of a 16-byte aligned output in tiles of `rounds` x kBlock
// vectors spread over the grid (as the batched kernel; larger tiles measured
// faster checks of the 4 GiB tensor written: 1585 -> 1507 us), then the
// n - nvec V ragged tail elements, one per thread of the first threads of
// the grid.  kNarrow:
// every block index and byte offset of the launch fits 32 bits (the launch
// checks), so the loop counts, the Philox counter and the addresses are
// 32-bit (the counter's high word is 0).
template <int DIST, int DT, bool kNarrow, bool kNT>
__global__ __launch_bounds__(kBlock) void synth_vec_kernel(SynthParams p, uint64_t nvec, uint64_t n,
                                                           u32x4 *__restrict__ out, uint32_t rounds) {
  prepare_distribution<DIST>();
  constexpr int E = PerBlock<DIST, DT>::E;
  constexpr int V = DT == SV_U8 ? 16 : DT == SV_BF16 || DT == SV_F16 ? 8 : 4;   // elements per 16-byte vector
  constexpr int B = V / E;                   // Philox blocks per vector
  using Idx = typename std::conditional<kNarrow, uint32_t, uint64_t>::type;
  const Idx gid = (Idx)blockIdx.x * kBlock + threadIdx.x;
  const Idx tile = (Idx)rounds * kBlock;
  const Idx c0 = (Idx)p.c0;
  SynthParams q = p;
  if constexpr (DIST == SV_NORMAL) q.mean = in_vgpr(p.mean);   // the addend of mean + std z
  const auto vector_at = [&](Idx u) {
    uint32_t v[V];
#pragma unroll
    for (int b = 0; b < B; ++b) values_of<DIST, DT>(q, (uint64_t)(c0 + u * B + b), v + b * E);
    u32x4 o;
    if constexpr (DT == SV_BF16) {
      o.x = bf16_pair<DIST>(v[0], v[1]);
      o.y = bf16_pair<DIST>(v[2], v[3]);
      o.z = bf16_pair<DIST>(v[4], v[5]);
      o.w = bf16_pair<DIST>(v[6], v[7]);
    } else if constexpr (DT == SV_F16) {
      static_assert(DIST == SV_UNIFORM || DIST == SV_NORMAL, "fp16 values here are never NaN");
      o.x = narrow_pair_not_nan<SV_F16>(v[0], v[1]);
      o.y = narrow_pair_not_nan<SV_F16>(v[2], v[3]);
      o.z = narrow_pair_not_nan<SV_F16>(v[4], v[5]);
      o.w = narrow_pair_not_nan<SV_F16>(v[6], v[7]);
    } else if constexpr (DT == SV_U8) {
#pragma unroll
      for (int k = 0; k < 4; ++k) o[k] = v[4 * k] | (v[4 * k + 1] << 8) | (v[4 * k + 2] << 16) | (v[4 * k + 3] << 24);
    } else {
      o = u32x4{v[0], v[1], v[2], v[3]};
    }
    store_vec<kNT>(out, u, o);
  };
  for (Idx t0 = (Idx)blockIdx.x * tile; t0 < (Idx)nvec; t0 += (Idx)gridDim.x * tile) {
    if (t0 + tile <= (Idx)nvec) {
      // a whole tile: a uniform trip count and no per-lane bound
      for (uint32_t r = 0; r < rounds; ++r) vector_at(t0 + (Idx)r * kBlock + threadIdx.x);
    } else {
      for (uint32_t r = 0; r < rounds; ++r) {
        const Idx u = t0 + (Idx)r * kBlock + threadIdx.x;
        if (u >= (Idx)nvec) break;
        vector_at(u);
      }
    }
  }
  const uint64_t i = nvec * V + (uint64_t)gid;
  if (i < n) {
    const uint64_t g = p.e0 + i;
    uint32_t v[E];
    values_of<DIST, DT>(p, g / E, v);
    store_elem<DIST, DT>(out, i, v[g % E]);
  }
}

// Special values, fp32, 16-byte aligned output, window starting on a block:
// the path of the special-value stream.  One vector = one normal block.  A
// vector with candidates (each element is one with probability gate / 256)
// needs the class block as well; rather than every lane computing one
// whenever any lane of its wave needs it, each lane holds its next kGroup
// vectors in registers while the wave lists their candidate vectors in LDS
// (the vector's offset in the tile, its four gate bytes and its normal
// values; about 13 % of the vectors on the special-value stream); then the
// wave's lanes take the listed vectors 64 at a time, one class block each,
// and overwrite the special elements in LDS; each lane reads its listed
// vectors back and stores all kGroup of them once, in order.  kGroup = 6
// lists about 51 vectors on that stream, so one pass over the list nearly
// always covers it and few of its lanes idle.  (Storing the candidate
// vectors late, when a ring of them filled up, measured much slower: cache
// lines written in two pieces far apart in time; storing them twice, with
// normal values first, wrote 1.33 times the bytes.)  Loops are uniform across
// the wave (lanes past the end only compute), so every lane takes part in
// every pass over the list.
#ifndef SV_SPECIAL_GROUP
#define SV_SPECIAL_GROUP 6
#endif
constexpr uint32_t kGroup = SV_SPECIAL_GROUP;   // vectors a lane holds before their candidates are overlaid
#ifndef SV_SPECIAL_LIST
#define SV_SPECIAL_LIST 128
#endif
// List entries per wave (32 bytes each).  Listing a wave's next 64 vectors
// when the list cannot take all of its candidates, each candidate computes its
// class block itself instead: slower, but only for mixes in which most
// vectors hold a candidate.  The special-value stream lists about 51 per
// group of six vectors per lane, 11 standard deviations below 128.
constexpr uint32_t kSpecialList = SV_SPECIAL_LIST;

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// The class thresholds as 32-bit compares: a class word x is at or above
// threshold t (at most 2^32) iff t < 2^32 and x >= t.
struct SpecialClasses {
  uint32_t nan, inf, den, zero;
  bool nan_all, inf_all, den_all, zero_all;   // t = 2^32: no word reaches it
};

__device__ __forceinline__ SpecialClasses special_classes(const SynthParams &p) {
  const auto lo = [](uint64_t t) { return (uint32_t)(t > 0xFFFFFFFFull ? 0xFFFFFFFFull : t); };
  return SpecialClasses{lo(p.t_nan), lo(p.t_inf), lo(p.t_den), lo(p.t_zero),
                        p.t_nan > 0xFFFFFFFFull, p.t_inf > 0xFFFFFFFFull, p.t_den > 0xFFFFFFFFull,
                        p.t_zero > 0xFFFFFFFFull};
}

__device__ __forceinline__ bool at_or_above(uint32_t x, uint32_t t, bool all) { return !all && x >= t; }

// A candidate element whose class word is x: its special value, or nv (its
// normal value) when x is at or above the last threshold -- special_overlay's
// values, with selects in place of branches.
__device__ __forceinline__ uint32_t special_or_keep(const SpecialClasses &c, uint32_t x, uint32_t nv) {
  const uint32_t r = x * kPayloadHash;
  const uint32_t m = r & 0x007FFFFFu;
  uint32_t e = at_or_above(x, c.den, c.den_all) ? 0u : (m > 1u ? m : 1u);      // zero : denormal
  e = at_or_above(x, c.inf, c.inf_all) ? e : 0x7F800000u;                     // Inf
  e = at_or_above(x, c.nan, c.nan_all) ? e : (0x7FC00000u | (r & 0x003FFFFFu));   // NaN
  return at_or_above(x, c.zero, c.zero_all) ? nv : ((r & 0x80000000u) | e);
}

// The four gate bytes of a normal block, element k in byte k: two byte
// permutes (v_perm_b32 picks bytes 0-3 of its second operand with selectors
// 0-3, of its first with 4-7, and 0x0C gives a zero byte) and an OR.
__device__ __forceinline__ uint32_t gate_bytes(const u32x4 &w) {
  return __builtin_amdgcn_perm(w.y, w.x, 0x0C0C0400u) | __builtin_amdgcn_perm(w.w, w.z, 0x04000C0Cu);
}

// The final values of a vector with normal values x, gate bytes b and class
// block q.
__device__ __forceinline__ u32x4 overlay_vector(const SpecialClasses &cls, uint32_t gate, const u32x4 &q,
                                                uint32_t b, u32x4 x) {
  x.x = (b & 0xFFu) < gate ? special_or_keep(cls, q.x, x.x) : x.x;
  x.y = ((b >> 8) & 0xFFu) < gate ? special_or_keep(cls, q.y, x.y) : x.y;
  x.z = ((b >> 16) & 0xFFu) < gate ? special_or_keep(cls, q.z, x.z) : x.z;
  x.w = (b >> 24) < gate ? special_or_keep(cls, q.w, x.w) : x.w;
  return x;
}

// DT: fp32, bf16, fp16 or fp64 output.  The kernel works in units: one
// 16-byte vector for fp32 (one block) and for the 16-bit types (two blocks,
// eight elements), two vectors for fp64 (one block).  A lane's kGroup slots
// are normal blocks: kGroup units for fp32 and fp64; kGroup / 2 for the
// 16-bit types, slot g being half g % 2 of unit g / 2.  The list is one of
// blocks either way; for the 16-bit types the overlay pass leaves a listed
// block's four final values in the entry already converted (two words);
// fp64 widens the four fp32 values of every block as it stores them.
template <int DT, bool kNarrow, bool kNT>
__global__ __launch_bounds__(kBlock) void synth_special_kernel(SynthParams p, uint64_t nvec, uint64_t n,
                                                               u32x4 *__restrict__ out, uint32_t rounds) {
  load_sincos_table();
  using Idx = typename std::conditional<kNarrow, uint32_t, uint64_t>::type;
  constexpr uint32_t kBpv = DT == SV_BF16 || DT == SV_F16 ? 2 : 1;   // normal blocks per unit
  constexpr uint32_t kVecs = kGroup / kBpv;         // units per lane per group
  static_assert(kGroup % kBpv == 0, "a group holds whole vectors");
  constexpr int kWaves = kBlock / kWave;
  constexpr uint32_t kSlots = kSpecialList;       // list entries per wave
  // entry: [0] a listed block's normal values, then its final ones; [1].xy
  // its offset in the tile (in blocks) and its gate bytes (one address
  // serves both)
  __shared__ u32x4 list[kWaves][kSlots][2];
  const uint32_t lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
  u32x4 (*lw)[2] = list[wave];
  const Key key{p.k0, p.k1, p.s0, p.s1};
  const SpecialClasses cls = special_classes(p);
  const uint32_t gate = p.gate;
  const float mean = in_vgpr(p.mean);
  const Idx tile = (Idx)rounds * kBlock;          // rounds: a multiple of kVecs
  const Idx c0 = (Idx)p.c0;
  const auto group = [&](Idx t0, uint32_t r0, auto whole_tile) {
    constexpr bool kWhole = decltype(whole_tile)::value;   // every vector of the tile is in range
    u32x4 v[kGroup];
    u32x4 *ent[kGroup];                           // the listed blocks' entries
    bool listed[kGroup];
    bool done[kGroup];                            // 16-bit types: overlaid and converted here (list full)
    uint32_t count = 0;                           // wave-uniform
#pragma unroll
    for (uint32_t g = 0; g < kGroup; ++g) {
      const uint32_t vo = (r0 + g / kBpv) * kBlock + threadIdx.x;   // the vector's offset in the tile
      const uint32_t off = vo * kBpv + g % kBpv;                     // the block's
      const Idx u = t0 + (Idx)vo;
      const Idx blk = c0 + t0 * (Idx)kBpv + (Idx)off;
      const u32x4 w = philox_block(key, (uint64_t)blk);
      float zc0, zs0, zc1, zs1;
      box_muller(w.x, w.y, zc0, zs0);
      box_muller(w.z, w.w, zc1, zs1);
      v[g] = u32x4{as_u32(__builtin_fmaf(p.std, zc0, mean)), as_u32(__builtin_fmaf(p.std, zs0, mean)),
                   as_u32(__builtin_fmaf(p.std, zc1, mean)), as_u32(__builtin_fmaf(p.std, zs1, mean))};
      const uint32_t low = min(min(w.x & 0xFFu, w.y & 0xFFu), min(w.z & 0xFFu, w.w & 0xFFu));
      listed[g] = low < gate && (kWhole || u < (Idx)nvec);
      done[g] = false;
      const uint64_t m = __ballot(listed[g]);
      const uint32_t nm = (uint32_t)__popcll(m);
      if (count + nm <= kSlots) {
        ent[g] = lw[__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, count))];
        if (listed[g]) {
          ent[g][0] = v[g];
          *(u32x2 *)&ent[g][1] = u32x2{off, gate_bytes(w)};
        }
        count += nm;
      } else if (listed[g]) {
        // the list is full (a mix with many candidates): this block's class block here
        const u32x4 q = philox_block(key, kSpecialClassBlocks + (uint64_t)blk);
        v[g] = overlay_vector(cls, gate, q, gate_bytes(w), v[g]);
        if constexpr (DT == SV_BF16 || DT == SV_F16) {
          v[g].x = narrow_pair<DT>(v[g].x, v[g].y);
          v[g].y = narrow_pair<DT>(v[g].z, v[g].w);
          done[g] = true;
        }
        listed[g] = false;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    for (uint32_t base = 0; base < count; base += kWave) {   // the listed blocks, one per lane
      const uint32_t e = base + lane;
      if (e < count) {
        const u32x2 k = *(const u32x2 *)&lw[e][1];
        const u32x4 q = philox_block(key, kSpecialClassBlocks + (uint64_t)(Idx)(c0 + t0 * (Idx)kBpv + (Idx)k.x));
        const u32x4 f = overlay_vector(cls, gate, q, k.y, lw[e][0]);
        if constexpr (DT == SV_F32 || DT == SV_F64)
          lw[e][0] = f;
        else
          *(u32x2 *)&lw[e][0] = u32x2{narrow_pair<DT>(f.x, f.y), narrow_pair<DT>(f.z, f.w)};
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (uint32_t j = 0; j < kVecs; ++j) {
      const Idx u = t0 + (Idx)((r0 + j) * kBlock + threadIdx.x);
      u32x4 o;
      if constexpr (DT == SV_F32) {
        if (listed[j]) v[j] = ent[j][0];
        o = v[j];
      } else if constexpr (DT == SV_F64) {
        if (listed[j]) v[j] = ent[j][0];
        const uint64_t w0 = widen_f32_bits(v[j].x), w1 = widen_f32_bits(v[j].y);
        const uint64_t w2 = widen_f32_bits(v[j].z), w3 = widen_f32_bits(v[j].w);
        if (kWhole || u < (Idx)nvec)
          store_vec<kNT>(out, 2 * u, u32x4{(uint32_t)w0, (uint32_t)(w0 >> 32), (uint32_t)w1, (uint32_t)(w1 >> 32)});
        o = u32x4{(uint32_t)w2, (uint32_t)(w2 >> 32), (uint32_t)w3, (uint32_t)(w3 >> 32)};
      } else {
        u32x2 h[2];
#pragma unroll
        for (uint32_t b = 0; b < 2; ++b) {
          const uint32_t g = 2 * j + b;
          h[b] = u32x2{narrow_pair_not_nan<DT>(v[g].x, v[g].y), narrow_pair_not_nan<DT>(v[g].z, v[g].w)};
          if (done[g]) h[b] = u32x2{v[g].x, v[g].y};
          if (listed[g]) h[b] = *(const u32x2 *)&ent[g][0];
        }
        o = u32x4{h[0].x, h[0].y, h[1].x, h[1].y};
      }
      if (kWhole || u < (Idx)nvec) store_vec<kNT>(out, DT == SV_F64 ? 2 * u + 1 : u, o);
    }
    // the list is rewritten by the next group only after every lane has read it
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  };
  for (Idx t0 = (Idx)blockIdx.x * tile; t0 < (Idx)nvec; t0 += (Idx)gridDim.x * tile) {
    if (t0 + tile <= (Idx)nvec) {
      for (uint32_t r0 = 0; r0 < rounds; r0 += kVecs) group(t0, r0, std::true_type{});
    } else {
      for (uint32_t r0 = 0; r0 < rounds; r0 += kVecs) group(t0, r0, std::false_type{});
    }
  }
  // the ragged tail elements, one per thread of the first threads of the grid
  constexpr uint32_t kPerVec = 4 * kBpv;
  const uint64_t i = nvec * kPerVec + (uint64_t)blockIdx.x * kBlock + threadIdx.x;
  if (i < n) {
    const uint64_t g = p.e0 + i;
    uint32_t e[4];
    block_values<SV_SPECIAL>(p, g / 4, e);
    if constexpr (DT == SV_F32)
      ((uint32_t *)out)[i] = e[g % 4];
    else if constexpr (DT == SV_F64)
      ((uint64_t *)out)[i] = widen_f32_bits(e[g % 4]);
    else if constexpr (DT == SV_BF16)
      ((uint16_t *)out)[i] = (uint16_t)bf16_rne(e[g % 4]);
    else
      ((uint16_t *)out)[i] = (uint16_t)f16_rne(e[g % 4]);
  }
}

// Special values into a 16-byte aligned output whose window starts on a
// block, through synth_special_kernel: whole groups of vectors per thread in
// a tile; 32-bit indices where every block index and vector offset fits.
template <int DT>
static hipError_t launch_special(const SynthParams &p, uint64_t n, void *out, int cus, bool nt, hipStream_t stream) {
  constexpr uint64_t kBpv = DT == SV_BF16 || DT == SV_F16 ? 2 : 1, V = 4 * kBpv, kVecs = kGroup / kBpv;
  constexpr uint64_t kVpu = DT == SV_F64 ? 2 : 1;   // 16-byte vectors per unit
  const uint64_t max_blocks = (uint64_t)cus * SV_SYNTH_BLOCKS_PER_CU;
  const uint64_t nvec = n / V;
  const uint32_t rounds = synth_tile_rounds(nvec, cus);
  const uint32_t r4 = (uint32_t)((rounds + kVecs - 1) / kVecs * kVecs);
  const uint64_t tile4 = (uint64_t)r4 * kBlock;
  const uint64_t blocks4 = std::max<uint64_t>(std::min<uint64_t>((nvec + tile4 - 1) / tile4, max_blocks),
                                              (n - nvec * V + kBlock - 1) / kBlock);   // the tail needs < V threads
  const bool narrow4 = p.c0 + (nvec + tile4) * kBpv < (1ull << 32) &&
                       (blocks4 * tile4 + nvec) * kBpv * kVpu < (1ull << 32);
  const dim3 g4((unsigned)blocks4), b4(kBlock);
  if (narrow4 && nt)
    hipLaunchKernelGGL((synth_special_kernel<DT, true, true>), g4, b4, 0, stream, p, nvec, n, (u32x4 *)out, r4);
  else if (narrow4)
    hipLaunchKernelGGL((synth_special_kernel<DT, true, false>), g4, b4, 0, stream, p, nvec, n, (u32x4 *)out, r4);
  else if (nt)
    hipLaunchKernelGGL((synth_special_kernel<DT, false, true>), g4, b4, 0, stream, p, nvec, n, (u32x4 *)out, r4);
  else
    hipLaunchKernelGGL((synth_special_kernel<DT, false, false>), g4, b4, 0, stream, p, nvec, n, (u32x4 *)out, r4);
  return hipGetLastError();
}

// Every element, one per thread (outputs that are not 16-byte aligned).
template <int DIST, int DT>
__global__ __launch_bounds__(kBlock) void synth_elem_kernel(SynthParams p, uint64_t n, void *__restrict__ out) {
  prepare_distribution<DIST>();
  constexpr int E = PerBlock<DIST, DT>::E;
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride) {
    const uint64_t g = p.e0 + i;
    uint32_t v[E];
    values_of<DIST, DT>(p, g / E, v);
    store_elem<DIST, DT>(out, i, v[g % E]);
  }
}

template <int DIST, int DT>
static hipError_t launch_typed(const SynthParams &p0, uint64_t n, void *out, int cus, hipStream_t stream) {
  constexpr uint64_t V = DT == SV_U8 ? 16 : DT == SV_BF16 || DT == SV_F16 ? 8 : 4;
  const SynthParams &p = p0;
  const bool nt = n * (16 / V) >= SV_SYNTH_NT_BYTES;
  const uint64_t max_blocks = (uint64_t)cus * SV_SYNTH_BLOCKS_PER_CU;
  if (((uintptr_t)out & 15u) == 0 && p.e0 % PerBlock<DIST, DT>::E == 0) {
    const uint64_t nvec = n / V;
    constexpr uint64_t B = V / PerBlock<DIST, DT>::E;
    const uint32_t rounds = synth_tile_rounds(nvec, cus);   // vectors per thread in a tile, as for batches
    const uint64_t tile = (uint64_t)rounds * kBlock;
    const uint64_t tblocks = std::max<uint64_t>(std::min<uint64_t>((nvec + tile - 1) / tile, max_blocks),
                                                (n - nvec * V + kBlock - 1) / kBlock);   // the tail needs < V threads
    if constexpr (DIST == SV_SPECIAL) return launch_special<DT>(p, n, out, cus, nt, stream);
    const bool narrow = p.c0 + (nvec + tile) * B < (1ull << 32) && tblocks * tile + nvec < (1ull << 32);
    const dim3 g((unsigned)tblocks), b(kBlock);
    if (narrow && nt)
      hipLaunchKernelGGL((synth_vec_kernel<DIST, DT, true, true>), g, b, 0, stream, p, nvec, n, (u32x4 *)out, rounds);
    else if (narrow)
      hipLaunchKernelGGL((synth_vec_kernel<DIST, DT, true, false>), g, b, 0, stream, p, nvec, n, (u32x4 *)out, rounds);
    else if (nt)
      hipLaunchKernelGGL((synth_vec_kernel<DIST, DT, false, true>), g, b, 0, stream, p, nvec, n, (u32x4 *)out, rounds);
    else
      hipLaunchKernelGGL((synth_vec_kernel<DIST, DT, false, false>), g, b, 0, stream, p, nvec, n, (u32x4 *)out, rounds);
  } else {
    const uint64_t blocks = std::min<uint64_t>((n + kBlock - 1) / kBlock, max_blocks);
    hipLaunchKernelGGL((synth_elem_kernel<DIST, DT>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, p, n, out);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------ fp16, fp64, uint8, int64
// The same elements stored in the other types: fp16 bits, fp64 bits, the
// int64.  E elements per Philox block as above, except fp64 uniform (53
// random bits from a 64-bit word: E = 2) and uint8, whose range of at most
// 256 values takes one 32-bit word per element (E = 4; the multiply-shift is
// then biased by less than 2^-24).  A 16-byte vector holds V = 16 / itemsize
// elements; only fp64 normal has V < E (two of a block's four).
template <int DIST, int DT> struct Wide {
  static constexpr int E = (DIST == SV_UNIFORM && DT == SV_F64) ? 2
                           : (DIST == SV_INT_RANGE && DT == SV_U8) ? 4
                                                                   : DistTraits<DIST>::E;
  static constexpr int V = DT == SV_F16 ? 8 : DT == SV_U8 ? 16 : 2;
};

template <int DIST, int DT>
__device__ __forceinline__ uint64_t from_value32(uint32_t v) {
  if constexpr (DT == SV_F16 && (DIST == SV_UNIFORM || DIST == SV_NORMAL)) {   // never NaN: no NaN rule
    // The fp16 value is the rounding of the fp32 value: the empty asm keeps
    // the compiler from fusing the fp32 multiply-add before it and this
    // conversion into one mixed-precision fma that rounds once, to fp16.
    uint32_t b = v;
    asm("" : "+v"(b));
    return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)as_f32(b));
  }
  else if constexpr (DT == SV_F16) return f16_rne(v);
  else if constexpr (DT == SV_F64) return widen_f32_bits(v);
  else return v & 0xFFu;                       // (not reached for uint8: wide_block forms its values)
}

// The E stored values of Philox block `block`.
template <int DIST, int DT>
__device__ __forceinline__ void wide_block(const SynthParams &p, uint64_t block, uint64_t *v) {
  if constexpr ((DIST == SV_UNIFORM && DT == SV_F64) || (DIST == SV_INT_RANGE && DT == SV_I64)) {
    const u32x4 w = philox_block(Key{p.k0, p.k1, p.s0, p.s1}, block);
    const uint64_t r[2] = {((uint64_t)w.y << 32) | w.x, ((uint64_t)w.w << 32) | w.z};
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      if constexpr (DIST == SV_UNIFORM) {
        const double t = p.span64 * ((double)(r[k] >> 11) * 0x1p-53);
        v[k] = f64_bits(p.a64 + t);
      } else {
        v[k] = (uint64_t)p.lo + (p.range ? __umul64hi(r[k], p.range) : r[k]);
      }
    }
  } else if constexpr (DIST == SV_INT_RANGE && DT == SV_U8) {
    const u32x4 w = philox_block(Key{p.k0, p.k1, p.s0, p.s1}, block);
    const uint32_t lo = (uint32_t)p.lo, range = (uint32_t)p.range;   // range <= 256
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = lo + __umulhi(w[k], range);
  } else {
    constexpr int E = DistTraits<DIST>::E;
    uint32_t f[E];
    block_values<DIST>(p, block, f);
#pragma unroll
    for (int k = 0; k < E; ++k) v[k] = from_value32<DIST, DT>(f[k]);
  }
}

template <int DT>
__device__ __forceinline__ void store_wide(void *out, uint64_t i, uint64_t x) {
  if constexpr (DT == SV_F16) ((uint16_t *)out)[i] = (uint16_t)x;
  else if constexpr (DT == SV_U8) ((uint8_t *)out)[i] = (uint8_t)x;
  else ((uint64_t *)out)[i] = x;
}

template <int DIST, int DT>
__device__ __forceinline__ uint64_t wide_elem(const SynthParams &p, uint64_t g) {
  constexpr int E = Wide<DIST, DT>::E;
  uint64_t v[E];
  wide_block<DIST, DT>(p, g / E, v);
  return v[g % E];
}

// Groups of G 16-byte vectors, W = G V elements: one vector (G = 1) made of
// V / E whole blocks, or, where a vector holds fewer elements than a block
// (fp64 normal and special: V = 2, E = 4), the G = E / V vectors of one
// block, so that no Philox word is wasted.  Then the n - groups W ragged tail
// elements, one per thread of the first threads of the grid (the window
// starts on a block).
template <int DIST, int DT, bool kNT>
__global__ __launch_bounds__(kBlock) void synth_wide_vec_kernel(SynthParams p, uint64_t ngroups, uint64_t n,
                                                                u32x4 *__restrict__ out) {
  prepare_distribution<DIST>();
  constexpr int E = Wide<DIST, DT>::E, V = Wide<DIST, DT>::V;
  constexpr int G = V >= E ? 1 : E / V;
  constexpr int W = G * V;
  const uint64_t gid = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t g = gid; g < ngroups; g += stride) {
    uint64_t v[W];
    if constexpr (G == 1) {
#pragma unroll
      for (int b = 0; b < V / E; ++b) wide_block<DIST, DT>(p, p.c0 + g * (V / E) + b, v + b * E);
    } else {
      wide_block<DIST, DT>(p, p.c0 + g, v);
    }
#pragma unroll
    for (int j = 0; j < G; ++j) {
      const uint64_t *x = v + j * V;
      u32x4 o;
      if constexpr (DT == SV_F16) {
#pragma unroll
        for (int k = 0; k < 4; ++k) o[k] = (uint32_t)x[2 * k] | ((uint32_t)x[2 * k + 1] << 16);
      } else if constexpr (DT == SV_U8) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          o[k] = (uint32_t)x[4 * k] | ((uint32_t)x[4 * k + 1] << 8) | ((uint32_t)x[4 * k + 2] << 16) |
                 ((uint32_t)x[4 * k + 3] << 24);
      } else {
        o = u32x4{(uint32_t)x[0], (uint32_t)(x[0] >> 32), (uint32_t)x[1], (uint32_t)(x[1] >> 32)};
      }
      store_vec<kNT>(out, g * G + j, o);
    }
  }
  const uint64_t i = ngroups * W + gid;
  if (i < n) store_wide<DT>(out, i, wide_elem<DIST, DT>(p, p.e0 + i));
}

template <int DIST, int DT>
__global__ __launch_bounds__(kBlock) void synth_wide_elem_kernel(SynthParams p, uint64_t n, void *__restrict__ out) {
  prepare_distribution<DIST>();
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride)
    store_wide<DT>(out, i, wide_elem<DIST, DT>(p, p.e0 + i));
}

template <int DIST, int DT>
static hipError_t launch_wide(const SynthParams &p0, uint64_t n, void *out, int cus, hipStream_t stream) {
  constexpr uint64_t E = Wide<DIST, DT>::E, V = Wide<DIST, DT>::V;
  const SynthParams &p = p0;
  const bool nt = n * (16 / V) >= SV_SYNTH_NT_BYTES;
  constexpr uint64_t W = V >= E ? V : E;          // elements per group of vectors
  const uint64_t max_blocks = (uint64_t)cus * SV_SYNTH_BLOCKS_PER_CU;
  if constexpr (DIST == SV_SPECIAL && (DT == SV_F16 || DT == SV_F64))
    if (((uintptr_t)out & 15u) == 0 && p.e0 % 4 == 0) return launch_special<DT>(p, n, out, cus, nt, stream);
  if (((uintptr_t)out & 15u) == 0 && p.e0 % E == 0) {
    const uint64_t ngroups = n / W;
    const uint64_t threads = std::max<uint64_t>(ngroups, n - ngroups * W);   // the tail needs < W threads
    const uint64_t blocks = std::min<uint64_t>((threads + kBlock - 1) / kBlock, max_blocks);
    if (nt)
      hipLaunchKernelGGL((synth_wide_vec_kernel<DIST, DT, true>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, p,
                         ngroups, n, (u32x4 *)out);
    else
      hipLaunchKernelGGL((synth_wide_vec_kernel<DIST, DT, false>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, p,
                         ngroups, n, (u32x4 *)out);
  } else {
    const uint64_t blocks = std::min<uint64_t>((n + kBlock - 1) / kBlock, max_blocks);
    hipLaunchKernelGGL((synth_wide_elem_kernel<DIST, DT>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, p, n,
                       out);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------ permutation
// Element i = lo + pi(i), pi a bijection of [0, N): the word permutation
// G(x) = (Feistel(x) + K_10) mod 2^2h on the smallest even-bit domain 2^2h >=
// N, applied again until the word falls below N (cycle walking: i's own cycle
// returns to [0, N), after fewer than 4 steps on average as 2^2h < 4N).  Ten
// Feistel rounds map the h-bit halves (L, R) to (R, L xor (F(R xor K_r) mod
// 2^h)), F the lowbias32 integer hash (C. Wellons, hash-prospector, 2018).
// Feistel rounds alone are even permutations of the words, from which the
// walk does not reach every order of [0, N) equally often; the keyed
// rotation, odd for odd K_10, evens this out.  K_0 .. K_10 are the words of
// Philox blocks 0, 1 and 2 of the tensor's (seed, stream) sequence, which
// every thread forms once.  The walk lengths differ from element to element
// (geometric, mean below 4): a lane whose element has landed stores it and
// takes its next element at once, so that a wave does not wait on its
// slowest lane for each element (the longest of 64 walks averages ~16 steps).
__device__ __forceinline__ uint32_t lowbias32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

template <int DT>
__global__ __launch_bounds__(kBlock) void synth_perm_kernel(SynthParams p, uint64_t n, void *__restrict__ out) {
  const Key key{p.k0, p.k1, p.s0, p.s1};
  const u32x4 b0 = philox_block(key, 0), b1 = philox_block(key, 1), b2 = philox_block(key, 2);
  const uint32_t k[11] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w, b2.x, b2.y, b2.z};
  const uint32_t h = p.half;
  const uint32_t mask = (1u << h) - 1u;
  const uint64_t words = (1ull << (2u * h)) - 1u;
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x;   // this lane's element
  uint64_t x = p.e0 + i;                                     // its word so far
  bool live = i < n;
  // every walk returns below N (its element's own cycle does), and each lane
  // then moves on by `stride` until it passes n: every wave leaves the loop
  while (__any(live)) {
    if (live) {
      uint32_t l = (uint32_t)(x >> h), r = (uint32_t)x & mask;
#pragma unroll
      for (int rd = 0; rd < 10; ++rd) {
        const uint32_t t = l ^ (lowbias32(r ^ k[rd]) & mask);
        l = r;
        r = t;
      }
      x = ((((uint64_t)l << h) | r) + k[10]) & words;
      if (x < p.range) {
        const uint64_t v = (uint64_t)p.lo + x;
        if constexpr (DT == SV_U8) ((uint8_t *)out)[i] = (uint8_t)v;
        else if constexpr (DT == SV_I32) ((uint32_t *)out)[i] = (uint32_t)v;
        else ((uint64_t *)out)[i] = v;
        i += stride;
        live = i < n;
        x = p.e0 + i;
      }
    }
  }
}

template <int DT>
static hipError_t launch_perm(const SynthParams &p, uint64_t n, void *out, int cus, hipStream_t stream) {
  const uint64_t blocks = std::min<uint64_t>((n + kBlock - 1) / kBlock, (uint64_t)cus * SV_SYNTH_BLOCKS_PER_CU);
  hipLaunchKernelGGL((synth_perm_kernel<DT>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, p, n, out);
  return hipGetLastError();
}

hipError_t launch_synth(int32_t dtype, int32_t dist, const SynthParams &p, uint64_t n, void *out, int cus,
                        hipStream_t stream) {
  switch (dist * 8 + dtype) {
    case SV_UNIFORM * 8 + SV_F32: return launch_typed<SV_UNIFORM, SV_F32>(p, n, out, cus, stream);
    case SV_UNIFORM * 8 + SV_BF16: return launch_typed<SV_UNIFORM, SV_BF16>(p, n, out, cus, stream);
    case SV_NORMAL * 8 + SV_F32: return launch_typed<SV_NORMAL, SV_F32>(p, n, out, cus, stream);
    case SV_NORMAL * 8 + SV_BF16: return launch_typed<SV_NORMAL, SV_BF16>(p, n, out, cus, stream);
    case SV_INT_RANGE * 8 + SV_I32: return launch_typed<SV_INT_RANGE, SV_I32>(p, n, out, cus, stream);
    case SV_SPECIAL * 8 + SV_F32: return launch_typed<SV_SPECIAL, SV_F32>(p, n, out, cus, stream);
    case SV_SPECIAL * 8 + SV_BF16: return launch_typed<SV_SPECIAL, SV_BF16>(p, n, out, cus, stream);
    case SV_UNIFORM * 8 + SV_F16: return launch_typed<SV_UNIFORM, SV_F16>(p, n, out, cus, stream);
    case SV_UNIFORM * 8 + SV_F64: return launch_wide<SV_UNIFORM, SV_F64>(p, n, out, cus, stream);
    case SV_NORMAL * 8 + SV_F16: return launch_typed<SV_NORMAL, SV_F16>(p, n, out, cus, stream);
    case SV_NORMAL * 8 + SV_F64: return launch_wide<SV_NORMAL, SV_F64>(p, n, out, cus, stream);
    case SV_SPECIAL * 8 + SV_F16: return launch_wide<SV_SPECIAL, SV_F16>(p, n, out, cus, stream);
    case SV_SPECIAL * 8 + SV_F64: return launch_wide<SV_SPECIAL, SV_F64>(p, n, out, cus, stream);
    case SV_INT_RANGE * 8 + SV_U8: return launch_typed<SV_INT_RANGE, SV_U8>(p, n, out, cus, stream);
    case SV_INT_RANGE * 8 + SV_I64: return launch_wide<SV_INT_RANGE, SV_I64>(p, n, out, cus, stream);
    case SV_PERMUTATION * 8 + SV_I32: return launch_perm<SV_I32>(p, n, out, cus, stream);
    case SV_PERMUTATION * 8 + SV_U8: return launch_perm<SV_U8>(p, n, out, cus, stream);
    case SV_PERMUTATION * 8 + SV_I64: return launch_perm<SV_I64>(p, n, out, cus, stream);
    default: return hipErrorInvalidValue;
  }
}

// ------------------------------------------------------------ diagnostics
__global__ __launch_bounds__(kBlock) void eval_transform_kernel(int32_t which, const uint32_t *__restrict__ in,
                                                                uint64_t n, uint32_t *__restrict__ out) {
  load_sincos_table();
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride) {
    if (which == SV_EVAL_F16) {
      out[i] = f16_rne(in[i]);
      continue;
    }
    if (which == SV_EVAL_BF16) {
      out[i] = bf16x2_rne_not_nan(in[i], 0u) & 0xFFFFu;
      continue;
    }
    const uint32_t k = in[i] & 0x00FFFFFFu;
    float v;
    if (which == SV_EVAL_LN) {
      v = ln_f32((float)(k + 1u) * 0x1p-24f);
    } else if (which == SV_EVAL_RADIUS) {
      v = bm_radius(k);
    } else {
      float sn, cs;
      sincos_2pi(k, sn, cs);
      v = which == SV_EVAL_SIN ? sn : cs;
    }
    out[i] = as_u32(v);
  }
}

hipError_t launch_eval_transform(int32_t which, const uint32_t *in, uint64_t n, uint32_t *out, int cus,
                                 hipStream_t stream) {
  const uint64_t blocks = std::min<uint64_t>((n + kBlock - 1) / kBlock, (uint64_t)cus * 8);
  hipLaunchKernelGGL(eval_transform_kernel, dim3((unsigned)blocks), dim3(kBlock), 0, stream, which, in, n, out);
  return hipGetLastError();
}

// ------------------------------------------------------------ batched
// Output vector u of one job: the B Philox blocks that cover it, then one
// 16-byte store, or element stores where the vector is partial or the
// output is not 16-byte aligned.
template <int DIST, int DT>
__device__ __forceinline__ void synth_vector(const SynthParams &p, void *out, uint64_t n, uint64_t u,
                                             bool vec_ok) {
  constexpr int E = PerBlock<DIST, DT>::E;
  constexpr int V = DT == SV_BF16 ? 8 : 4;
  constexpr int B = V / E;
  uint32_t v[V];
#pragma unroll
  for (int b = 0; b < B; ++b) values_of<DIST, DT>(p, u * B + b, v + b * E);
  if (vec_ok && (u + 1) * V <= n) {
    u32x4 o;
    if constexpr (DT == SV_BF16) {
      o.x = bf16_pair<DIST>(v[0], v[1]);
      o.y = bf16_pair<DIST>(v[2], v[3]);
      o.z = bf16_pair<DIST>(v[4], v[5]);
      o.w = bf16_pair<DIST>(v[6], v[7]);
    } else {
      o = u32x4{v[0], v[1], v[2], v[3]};
    }
    ((u32x4 *)out)[u] = o;
  } else {
#pragma unroll
    for (int j = 0; j < V; ++j)
      if (u * V + j < n) store_elem<DIST, DT>(out, u * V + j, v[j]);
  }
}

// Job holding tile t: the last job whose first tile is <= t (jobs without
// elements share their successor's first tile and are skipped by this rule).
__device__ __forceinline__ uint32_t find_job(const SynthJob *jobs, uint32_t njobs, uint64_t t) {
  uint32_t lo = 0, hi = njobs;
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) / 2;
    if (jobs[mid].tile_begin <= t) lo = mid; else hi = mid;
  }
  return lo;
}

// One tile of a job: `rounds` vectors per thread, kBlock apart.  A thread
// whose vectors are all whole and 16-byte aligned, in a job whose Philox
// counters fit 32 bits, takes the lean loop of the single-tensor kernel
// (32-bit counters, no per-vector checks); the others, at a job's end or for
// unaligned outputs, take the general one.
template <int DIST, int DT>
__device__ __forceinline__ void synth_tile(const SynthJob &job, uint64_t u0, uint32_t rounds, bool ok) {
  constexpr int E = PerBlock<DIST, DT>::E;
  constexpr int V = DT == SV_BF16 ? 8 : 4;
  constexpr uint32_t B = V / E;
  const uint64_t whole = job.n / V;
  if (ok && job.nvec * B < (1ull << 32) && u0 + (uint64_t)(rounds - 1) * kBlock < whole) {
    u32x4 *out = (u32x4 *)job.out;
    for (uint32_t r = 0; r < rounds; ++r) {
      const uint32_t u = (uint32_t)u0 + r * (uint32_t)kBlock;
      uint32_t v[V];
#pragma unroll
      for (uint32_t b = 0; b < B; ++b) values_of<DIST, DT>(job.p, (uint64_t)(u * B + b), v + b * E);
      u32x4 o;
      if constexpr (DT == SV_BF16) {
        o.x = bf16_pair<DIST>(v[0], v[1]);
        o.y = bf16_pair<DIST>(v[2], v[3]);
        o.z = bf16_pair<DIST>(v[4], v[5]);
        o.w = bf16_pair<DIST>(v[6], v[7]);
      } else {
        o = u32x4{v[0], v[1], v[2], v[3]};
      }
      out[u] = o;
    }
    return;
  }
  for (uint32_t r = 0; r < rounds; ++r) {
    const uint64_t u = u0 + (uint64_t)r * kBlock;
    if (u >= job.nvec) break;
    synth_vector<DIST, DT>(job.p, job.out, job.n, u, ok);
  }
}

// Tiles over the whole grid (the resident workgroups write neighbouring
// tiles); a workgroup searches the job table only when its next tile leaves
// the current job's tiles, and a tile holds `rounds` vectors per thread, so
// that the search and the loads of a job's parameters are rare.  Large tiles
// also measured faster checks of the data just written (bf16 batch of 64 x
// 2^24: 795 -> 694 us for 4 -> 32 vectors per thread); the host keeps at
// least SV_SYNTH_TILES_PER_CU tiles per CU so that small batches still fill
// the GPU.
__global__ __launch_bounds__(kBlock) void synth_batched_kernel(const SynthJob *__restrict__ jobs, uint32_t njobs,
                                                               uint64_t total_tiles, uint32_t rounds) {
  load_sincos_table();   // the jobs may draw normal values
  uint32_t j = 0;
  uint64_t lo = 1, hi = 0;           // tiles [lo, hi) belong to job j (none yet)
  for (uint64_t t = blockIdx.x; t < total_tiles; t += gridDim.x) {
    if (t < lo || t >= hi) {
      j = find_job(jobs, njobs, t);
      lo = jobs[j].tile_begin;
      hi = j + 1 < njobs ? jobs[j + 1].tile_begin : total_tiles;
    }
    const SynthJob &job = jobs[j];
    const uint64_t u0 = (t - lo) * rounds * kBlock + threadIdx.x;
    const bool ok = job.vec_ok != 0;
    switch (job.kind) {
      case SV_UNIFORM * 4 + SV_F32: synth_tile<SV_UNIFORM, SV_F32>(job, u0, rounds, ok); break;
      case SV_UNIFORM * 4 + SV_BF16: synth_tile<SV_UNIFORM, SV_BF16>(job, u0, rounds, ok); break;
      case SV_NORMAL * 4 + SV_F32: synth_tile<SV_NORMAL, SV_F32>(job, u0, rounds, ok); break;
      case SV_NORMAL * 4 + SV_BF16: synth_tile<SV_NORMAL, SV_BF16>(job, u0, rounds, ok); break;
      case SV_INT_RANGE * 4 + SV_I32: synth_tile<SV_INT_RANGE, SV_I32>(job, u0, rounds, ok); break;
      case SV_SPECIAL * 4 + SV_F32: synth_tile<SV_SPECIAL, SV_F32>(job, u0, rounds, ok); break;
      default: synth_tile<SV_SPECIAL, SV_BF16>(job, u0, rounds, ok); break;
    }
  }
}

hipError_t launch_synth_batched(const SynthJob *jobs, uint32_t njobs, uint64_t total_tiles, uint32_t rounds,
                                int cus, hipStream_t stream) {
  const uint64_t blocks = std::min<uint64_t>(total_tiles, (uint64_t)cus * SV_SYNTH_BLOCKS_PER_CU);
  hipLaunchKernelGGL(synth_batched_kernel, dim3((unsigned)blocks), dim3(kBlock), 0, stream, jobs, njobs,
                     total_tiles, rounds);
  return hipGetLastError();
}

}  // namespace sv

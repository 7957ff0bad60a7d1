// sv_perturb.hip -- candidate derivation for the synthetic workloads
// (sv_perturb).  Not part of the check: it builds candidates that are correct
// up to rounding, or carry known faults, so that the check has something to
// find.  One Philox block per element under the step's own substream: the
// first word selects the element, the top bit of the second word picks the
// direction and the second word the NaN payload mask, the top 24 bits of the
// third word give the scale variate.
#include "sv_device.h"
#include "sv_internal.h"

namespace sv {

template <int DT>
__device__ __forceinline__ uint64_t load_bits(const void *a, uint64_t i) {
  if constexpr (DT == SV_BF16 || DT == SV_F16) return ((const uint16_t *)a)[i];
  else if constexpr (DT == SV_U8) return ((const uint8_t *)a)[i];
  else if constexpr (DT == SV_F64 || DT == SV_I64) return ((const uint64_t *)a)[i];
  else return ((const uint32_t *)a)[i];
}

template <int DT>
__device__ __forceinline__ void store_bits(void *a, uint64_t i, uint64_t v) {
  if constexpr (DT == SV_BF16 || DT == SV_F16) ((uint16_t *)a)[i] = (uint16_t)v;
  else if constexpr (DT == SV_U8) ((uint8_t *)a)[i] = (uint8_t)v;
  else if constexpr (DT == SV_F64 || DT == SV_I64) ((uint64_t *)a)[i] = v;
  else ((uint32_t *)a)[i] = (uint32_t)v;
}

// float-typed element <-> fp32 (bf16 and fp16 widen exactly; narrowing rounds to nearest even)
template <int DT>
__device__ __forceinline__ float widen(uint64_t b) {
  if constexpr (DT == SV_BF16) return as_f32((uint32_t)b << 16);
  else if constexpr (DT == SV_F16) return f16_widen((uint32_t)b);
  else return as_f32((uint32_t)b);
}
template <int DT>
__device__ __forceinline__ uint64_t narrow(float x) {
  if constexpr (DT == SV_BF16) return bf16_rne(as_u32(x));
  else if constexpr (DT == SV_F16) return f16_rne(as_u32(x));
  else return as_u32(x);
}

template <int DT>
__device__ __forceinline__ uint64_t derive(const PerturbParams &p, uint64_t i, uint64_t y) {
  if (p.op == SV_OP_COPY) return y;
  const u32x4 w = philox_block(Key{p.k0, p.k1, p.s0, p.s1}, i);
  if (!((uint64_t)w.x < p.threshold)) return y;
  const bool up = (w.y >> 31) != 0u;
  if (p.op == SV_OP_ULP) {
    if constexpr (DT == SV_BF16) return next_bf16((uint32_t)y, up);
    else if constexpr (DT == SV_F16) return next_f16((uint32_t)y, up);
    else if constexpr (DT == SV_F64) return next_f64(y, up);
    else return next_f32((uint32_t)y, up);
  }
  if constexpr (DT == SV_F32 || DT == SV_BF16) {
    if (p.op == SV_OP_SCALE) {
      const float U = unit24(w.z);
      const float two = 2.0f * p.value;
      const float u = two * U - p.value;
      const float s = 1.0f + u;
      return narrow<DT>(widen<DT>(y) * s);
    }
    // SPECIAL_FLIP
    if constexpr (DT == SV_BF16) {
      const uint32_t mag = (uint32_t)y & 0x7FFFu;
      if (mag == 0u) return y ^ 0x8000u;
      if (mag > 0x7F80u) {
        const uint32_t m = w.y & 0x3Fu;
        return y ^ (m ? m : 1u);
      }
      return y;
    } else {
      const uint32_t mag = (uint32_t)y & 0x7FFFFFFFu;
      if (mag == 0u) return y ^ 0x80000000u;
      if (mag > 0x7F800000u) {
        const uint32_t m = w.y & 0x003FFFFFu;
        return y ^ (m ? m : 1u);
      }
      return y;
    }
  }
  return y;                                     // not reached: the host admits these steps only for fp32 / bf16
}

template <int DT>
__global__ __launch_bounds__(kBlock) void perturb_elem_kernel(PerturbParams p, uint64_t n,
                                                              const void *__restrict__ ref, void *cand) {
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride)
    store_bits<DT>(cand, i, derive<DT>(p, i, load_bits<DT>(ref, i)));
}

template <int DT>
__global__ __launch_bounds__(kBlock) void perturb_index_kernel(PerturbParams p, const uint64_t *__restrict__ idx,
                                                               uint64_t nidx, const void *ref, void *cand) {
  const uint64_t k = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
  if (k >= nidx) return;
  const uint64_t i = idx[k];
  const uint64_t y = load_bits<DT>(ref, i);
  uint64_t out;
  if (p.op == SV_OP_SET_AT) {
    out = DT == SV_BF16 || DT == SV_F16 ? (p.bits & 0xFFFFu) : DT == SV_U8 ? (p.bits & 0xFFu) : p.bits;
  } else if constexpr (DT == SV_I32 || DT == SV_U8 || DT == SV_I64) {
    out = y + 1u;                                   // FAULT_AT on integers, wrapping in their width
  } else if constexpr (DT == SV_F64) {
    // FAULT_AT in fp64.  x + (1 + |x|) has two NaN operands when x is a NaN,
    // and which one a sum returns is not fixed: the result is |x| quieted;
    // -Inf + Inf is the invalid operation's NaN, sign set, no payload
    const double x = bits_f64(y);
    const double t = 1.0 + fabs(x);
    out = __builtin_isnan(x) ? ((y & 0x7FFFFFFFFFFFFFFFull) | 0x0008000000000000ull)
          : x == -__builtin_inf() ? 0xFFF8000000000000ull : f64_bits(x + t);
  } else if (p.op == SV_OP_ADD_AT) {
    out = narrow<DT>(widen<DT>(y) + p.value);
  } else {
    // FAULT_AT: always outside any sane tolerance; NaN and -Inf as for fp64
    const float x = widen<DT>(y);
    const float r = __builtin_isnan(x) ? as_f32((as_u32(x) & 0x7FFFFFFFu) | 0x00400000u)
                    : x == -__builtin_inff() ? as_f32(0xFFC00000u) : x + (1.0f + fabsf(x));
    out = narrow<DT>(r);
  }
  store_bits<DT>(cand, i, out);
}

template <template <int> class K, class... A>
static void dispatch_dtype(int32_t dtype, dim3 grid, hipStream_t stream, A... args) {
  switch (dtype) {
    case SV_F32: hipLaunchKernelGGL(K<SV_F32>::fn, grid, dim3(kBlock), 0, stream, args...); break;
    case SV_BF16: hipLaunchKernelGGL(K<SV_BF16>::fn, grid, dim3(kBlock), 0, stream, args...); break;
    case SV_I32: hipLaunchKernelGGL(K<SV_I32>::fn, grid, dim3(kBlock), 0, stream, args...); break;
    case SV_F16: hipLaunchKernelGGL(K<SV_F16>::fn, grid, dim3(kBlock), 0, stream, args...); break;
    case SV_F64: hipLaunchKernelGGL(K<SV_F64>::fn, grid, dim3(kBlock), 0, stream, args...); break;
    case SV_U8: hipLaunchKernelGGL(K<SV_U8>::fn, grid, dim3(kBlock), 0, stream, args...); break;
    default: hipLaunchKernelGGL(K<SV_I64>::fn, grid, dim3(kBlock), 0, stream, args...); break;
  }
}

template <int DT> struct ElemK { static constexpr auto fn = perturb_elem_kernel<DT>; };
template <int DT> struct IndexK { static constexpr auto fn = perturb_index_kernel<DT>; };

hipError_t launch_perturb_elementwise(int32_t dtype, const PerturbParams &p, uint64_t n, const void *ref,
                                      void *cand, int cus, hipStream_t stream) {
  if (!n) return hipSuccess;
  const uint64_t blocks = std::min<uint64_t>((n + kBlock - 1) / kBlock, (uint64_t)cus * 8);
  dispatch_dtype<ElemK>(dtype, dim3((unsigned)blocks), stream, p, n, ref, cand);
  return hipGetLastError();
}

hipError_t launch_perturb_indexed(int32_t dtype, const PerturbParams &p, const uint64_t *idx_dev, uint64_t nidx,
                                  const void *ref, void *cand, hipStream_t stream) {
  if (!nidx) return hipSuccess;
  const uint64_t blocks = (nidx + kBlock - 1) / kBlock;
  dispatch_dtype<IndexK>(dtype, dim3((unsigned)blocks), stream, p, idx_dev, nidx, ref, cand);
  return hipGetLastError();
}

}  // namespace sv

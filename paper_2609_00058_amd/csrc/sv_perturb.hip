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
__device__ __forceinline__ uint32_t load_bits(const void *a, uint64_t i) {
  if constexpr (DT == SV_BF16)
    return ((const uint16_t *)a)[i];
  else
    return ((const uint32_t *)a)[i];
}

template <int DT>
__device__ __forceinline__ void store_bits(void *a, uint64_t i, uint32_t v) {
  if constexpr (DT == SV_BF16)
    ((uint16_t *)a)[i] = (uint16_t)v;
  else
    ((uint32_t *)a)[i] = v;
}

// float-typed element <-> fp32 (bf16 widens exactly; narrowing rounds to nearest even)
template <int DT>
__device__ __forceinline__ float widen(uint32_t b) {
  return DT == SV_BF16 ? as_f32(b << 16) : as_f32(b);
}
template <int DT>
__device__ __forceinline__ uint32_t narrow(float x) {
  return DT == SV_BF16 ? bf16_rne(as_u32(x)) : as_u32(x);
}

template <int DT>
__device__ __forceinline__ uint32_t derive(const PerturbParams &p, uint64_t i, uint32_t y) {
  if (p.op == SV_OP_COPY) return y;
  const u32x4 w = philox_block(Key{p.k0, p.k1, p.s0, p.s1}, i);
  if (!((uint64_t)w.x < p.threshold)) return y;
  const bool up = (w.y >> 31) != 0u;
  if (p.op == SV_OP_ULP) return DT == SV_BF16 ? next_bf16(y, up) : next_f32(y, up);
  if (p.op == SV_OP_SCALE) {
    const float U = unit24(w.z);
    const float two = 2.0f * p.value;
    const float u = two * U - p.value;
    const float s = 1.0f + u;
    return narrow<DT>(widen<DT>(y) * s);
  }
  // SPECIAL_FLIP
  if constexpr (DT == SV_BF16) {
    const uint32_t mag = y & 0x7FFFu;
    if (mag == 0u) return y ^ 0x8000u;
    if (mag > 0x7F80u) {
      const uint32_t m = w.y & 0x3Fu;
      return y ^ (m ? m : 1u);
    }
    return y;
  } else {
    const uint32_t mag = y & 0x7FFFFFFFu;
    if (mag == 0u) return y ^ 0x80000000u;
    if (mag > 0x7F800000u) {
      const uint32_t m = w.y & 0x003FFFFFu;
      return y ^ (m ? m : 1u);
    }
    return y;
  }
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
  const uint32_t y = load_bits<DT>(ref, i);
  uint32_t out;
  if (p.op == SV_OP_SET_AT) {
    out = DT == SV_BF16 ? (p.bits & 0xFFFFu) : p.bits;
  } else if (p.op == SV_OP_ADD_AT) {
    out = narrow<DT>(widen<DT>(y) + p.value);
  } else if constexpr (DT == SV_I32) {
    out = y + 1u;                                   // FAULT_AT on integers, wrapping
  } else {
    const float x = widen<DT>(y);
    out = narrow<DT>(x + (1.0f + fabsf(x)));        // FAULT_AT: always outside any sane tolerance
  }
  store_bits<DT>(cand, i, out);
}

hipError_t launch_perturb_elementwise(int32_t dtype, const PerturbParams &p, uint64_t n, const void *ref,
                                      void *cand, int cus, hipStream_t stream) {
  if (!n) return hipSuccess;
  const uint64_t blocks = std::min<uint64_t>((n + kBlock - 1) / kBlock, (uint64_t)cus * 8);
  if (dtype == SV_BF16)
    hipLaunchKernelGGL(perturb_elem_kernel<SV_BF16>, dim3((unsigned)blocks), dim3(kBlock), 0, stream, p, n, ref,
                       cand);
  else if (dtype == SV_F32)
    hipLaunchKernelGGL(perturb_elem_kernel<SV_F32>, dim3((unsigned)blocks), dim3(kBlock), 0, stream, p, n, ref,
                       cand);
  else
    hipLaunchKernelGGL(perturb_elem_kernel<SV_I32>, dim3((unsigned)blocks), dim3(kBlock), 0, stream, p, n, ref,
                       cand);
  return hipGetLastError();
}

hipError_t launch_perturb_indexed(int32_t dtype, const PerturbParams &p, const uint64_t *idx_dev, uint64_t nidx,
                                  const void *ref, void *cand, hipStream_t stream) {
  if (!nidx) return hipSuccess;
  const uint64_t blocks = (nidx + kBlock - 1) / kBlock;
  if (dtype == SV_BF16)
    hipLaunchKernelGGL(perturb_index_kernel<SV_BF16>, dim3((unsigned)blocks), dim3(kBlock), 0, stream, p, idx_dev,
                       nidx, ref, cand);
  else if (dtype == SV_F32)
    hipLaunchKernelGGL(perturb_index_kernel<SV_F32>, dim3((unsigned)blocks), dim3(kBlock), 0, stream, p, idx_dev,
                       nidx, ref, cand);
  else
    hipLaunchKernelGGL(perturb_index_kernel<SV_I32>, dim3((unsigned)blocks), dim3(kBlock), 0, stream, p, idx_dev,
                       nidx, ref, cand);
  return hipGetLastError();
}

}  // namespace sv

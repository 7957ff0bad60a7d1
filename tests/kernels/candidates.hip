// Candidate kernels for the performance-stage tests: a kernel of known
// duration, an empty one, and a correct and a faulty elementwise kernel whose
// outputs the functional check must accept and reject.
#include <hip/hip_runtime.h>

extern "C" __global__ void sv_test_empty() {}

// Busy-waits `ticks` periods of the constant-rate wall clock (s_memrealtime).
extern "C" __global__ void sv_test_spin(unsigned long long ticks) {
  const unsigned long long t0 = wall_clock64();
  while (wall_clock64() - t0 < ticks) __builtin_amdgcn_s_sleep(2);
}

// z = a x + y (product and sum rounded separately).
extern "C" __global__ void sv_test_axpy(float *z, const float *x, const float *y, float a, unsigned long long n) {
  const unsigned long long i = (unsigned long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) z[i] = a * x[i] + y[i];
}

// The same with an off-by-one bound: the last element is never written.
extern "C" __global__ void sv_test_axpy_tail_bug(float *z, const float *x, const float *y, float a,
                                                 unsigned long long n) {
  const unsigned long long i = (unsigned long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i + 1 < n) z[i] = a * x[i] + y[i];
}

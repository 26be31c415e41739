// Engine clock probe: measurement support for the benchmark, not an op of
// the training step. One wave runs a chain of dependent fp32 FMAs between
// two reads of the shader clock counter (s_memtime) and of the constant
// 100 MHz real-time counter (s_memrealtime); their ratio is the clock the
// wave's compute unit ran at over the interval.

#include "common.h"
#include "kernels.h"

namespace tfd {

namespace {

__global__ __launch_bounds__(64) void clock_probe_kernel(uint64_t* counters, int64_t iterations) {
  const uint64_t c0 = __builtin_amdgcn_s_memtime();
  const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
  float x = (float)threadIdx.x;
  for (int64_t i = 0; i < iterations; ++i) x = __builtin_fmaf(x, 0.999999f, 1e-7f);
  const uint64_t c1 = __builtin_amdgcn_s_memtime();
  const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
  // lanes 0..2 store one word each (vector stores)
  const int l = threadIdx.x;
  if (l < 3) counters[l] = l == 0 ? c1 - c0 : l == 1 ? r1 - r0 : (uint64_t)__float_as_uint(x);
}

}  // namespace

hipError_t launch_clock_probe(uint64_t* counters, int64_t iterations, hipStream_t s) {
  hipLaunchKernelGGL(clock_probe_kernel, dim3(1), dim3(64), 0, s, counters, iterations);
  return hipGetLastError();
}

}  // namespace tfd

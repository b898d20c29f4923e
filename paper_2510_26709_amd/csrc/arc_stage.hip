// Staging of the step's projection V_t: the host generates it into a pinned,
// device-mapped buffer, and this kernel moves it into device memory on the
// context's stream (the first work of a step).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "arc_device.h"
#include "arc_internal.h"

namespace arc {
namespace {

__global__ void __launch_bounds__(256)
stage_projection_kernel(const float* __restrict__ src, float* __restrict__ dst, int64_t n) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < n) dst[e] = src[e];
}

}  // namespace

hipError_t launch_stage_projection(const float* src, float* dst, int64_t n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(stage_projection_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, stream, src,
                     dst, n);
  return hipGetLastError();
}

}  // namespace arc

// Device fill of the synthetic-gradient recipe (synth_core.h): the same bits
// as synth_fill_host.  Input generation only; not part of libarctopk.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "synth_core.h"

__global__ void __launch_bounds__(256)
synth_fill_kernel(synth_plan pl, int64_t t, void* out) {
  const int64_t total = (int64_t)pl.N * pl.d;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int32_t cur_i = -1;
  synth_keys k{};
  for (; e < total; e += stride) {
    const int32_t i = (int32_t)(e / pl.d);
    const int64_t j = e - (int64_t)i * pl.d;
    if (i != cur_i) {
      k = synth_step_keys(&pl, t, i);
      cur_i = i;
    }
    const float v = synth_value(&pl, &k, j);
    if (pl.out_bf16)
      static_cast<uint16_t*>(out)[e] = synth_to_bf16(v);
    else
      static_cast<float*>(out)[e] = v;
  }
}

// Fills out[N*d] (device memory) for step t on `stream`.  The plan's tables
// (seg_begin, scale) must be device pointers.  Returns a hipError_t value.
extern "C" int synth_fill_device(const synth_plan* pl, int64_t t, void* out,
                                 void* stream) {
  if (pl == nullptr || out == nullptr) return (int)hipErrorInvalidValue;
  int dev = 0, cus = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return (int)err;
  err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (err != hipSuccess) return (int)err;
  const int64_t total = (int64_t)pl->N * pl->d;
  int64_t blocks = (total + 255) / 256;
  const int64_t cap = (int64_t)(cus > 0 ? cus : 256) * 32;
  if (blocks > cap) blocks = cap;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(synth_fill_kernel, dim3((unsigned)blocks), dim3(256), 0,
                     (hipStream_t)stream, *pl, t, out);
  return (int)hipGetLastError();
}

/* Host fill of the synthetic-gradient recipe (synth_core.h).  Input
 * generation only; shared by the tests, the benchmark and the oracle's
 * inputs.  Holds none of the compressor's arithmetic. */
#include <stdint.h>

#include "synth_core.h"

/* Values of workers [i0, i1) at coordinates [j0, j1) of step t into out
 * (row stride ld elements; binary32 or bf16 per plan->out_bf16). */
int synth_fill_host(const synth_plan *pl, int64_t t, int32_t i0, int32_t i1,
                    int64_t j0, int64_t j1, void *out, int64_t ld) {
  if (pl == 0 || out == 0 || i0 < 0 || i1 > pl->N || i0 > i1 || j0 < 0 ||
      j1 > pl->d || j0 > j1 || ld < j1 - j0)
    return 1;
  for (int32_t i = i0; i < i1; ++i) {
    const synth_keys k = synth_step_keys(pl, t, i);
#pragma omp parallel for schedule(static)
    for (int64_t j = j0; j < j1; ++j) {
      const float v = synth_value(pl, &k, j);
      const int64_t at = (int64_t)(i - i0) * ld + (j - j0);
      if (pl->out_bf16)
        ((uint16_t *)out)[at] = synth_to_bf16(v);
      else
        ((float *)out)[at] = v;
    }
  }
  return 0;
}

/* n standard normals from stream (seed, stream, 0, 0), counters 0..n-1:
 * used for the per-tensor / per-coordinate LogNormal scale tables. */
int synth_normals_host(uint64_t seed, uint64_t stream, int64_t n, float *out) {
  if (out == 0 || n < 0) return 1;
  const uint64_t key = synth_key(seed, stream, 0u, 0u);
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < n; ++j) out[j] = synth_normal(key, (uint64_t)j);
  return 0;
}

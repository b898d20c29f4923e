// General sketch kernel: the same streaming stage as the vectorised kernels
// (EF21M momentum (11a), Delta = h_t - g_{t-1}, per-worker sketch of Alg. 1)
// for row groups the 16-byte kernels cannot take: any row width, any r up to
// ARC_MAX_R, element-aligned pointers, and a ragged last row.
//
// One wave per (row group, worker); a group's rows may lie `stride` rows
// apart (vectorised groups, taken here when the pointers are misaligned).
// Each 32-column chunk of the group's
// 64 x 32 tile is loaded with one element per lane (two rows of 32 columns
// per instruction, coalesced), 24 loads in flight per pass of 16 rows; Delta
// goes to LDS, and so do the chunk's 32 rows of V (transposed to [k][j]).
// Lane p then runs its row's r chains over the chunk in ascending column
// order, its partial sums kept in LDS between chunks.  The arithmetic is the
// same as the vectorised kernels', in the same order, so both produce the
// same bits.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "arc_device.h"
#include "arc_internal.h"
#include "libarctopk.h"

namespace arc {
namespace {

constexpr int kGenChunk = 32;       // columns per chunk
constexpr int kGenPitch = kGenChunk + 1;  // LDS row pitch (floats), conflict-free row reads
constexpr int kGenRowsPerPass = 16;  // rows loaded per pass: 8 instructions x 2 rows

// norm != 0 (r = 1): the chain is the row's squared norm, fmaf(Delta, Delta,
// s), for the Top-K comparison compressor; V is unused.
template <bool BF16>
__global__ void __launch_bounds__(kWave)
sketch_general_kernel(const void* __restrict__ grad, float* __restrict__ h,
                      const float* __restrict__ g, const float* __restrict__ V,
                      const RowGroup* __restrict__ groups, float* __restrict__ S,
                      int64_t d, int64_t m, int32_t r, float eta, float a, int32_t norm) {
  __shared__ float tile[kWave * kGenPitch];
  extern __shared__ float dyn[];
  float* acc = dyn;              // [r][64] partial sums
  float* vl = dyn + r * kWave;   // [r][32] this chunk's rows of V
  const RowGroup grp = groups[blockIdx.x];
  const int lane = threadIdx.x;
  const int32_t i = blockIdx.y;
  const int64_t n = grp.cols;
  const int32_t rows = grp.rows;
  const int64_t row_step = (int64_t)grp.stride * n;  // elements between local rows
  const int64_t base = (int64_t)i * d + grp.elem_off;
  const float* Vg = V + grp.v_off;
  const int half = lane >> 5;            // row of the pair this lane loads
  const int cl = lane & (kGenChunk - 1);  // column within the chunk
  for (int32_t k = 0; k < r; ++k) acc[k * kWave + lane] = 0.0f;

  // A one-row group holds only the last row's values (a ragged tail row).
  const int64_t span = rows == 1 ? grp.last_len : n;
  for (int64_t c0 = 0; c0 < span; c0 += kGenChunk) {
    const int cw = (int)(span - c0 < kGenChunk ? span - c0 : kGenChunk);
    if (!norm) {
      for (int t = lane; t < r * kGenChunk; t += kWave) {
        const int k = t / kGenChunk, j = t - k * kGenChunk;
        vl[t] = Vg[(c0 + (j < cw ? j : cw - 1)) * r + k];
      }
    }
    for (int pass = 0; pass * kGenRowsPerPass < rows; ++pass) {
      float xv[8], hv[8], gv[8];
      bool ok[8];
      int64_t e[8];
      // Every lane loads; a lane without an element of the group loads the
      // group's first element instead (always present) and discards it.
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int l = pass * kGenRowsPerPass + u * 2 + half;
        const int64_t len = l == rows - 1 ? grp.last_len : n;
        ok[u] = l < rows && cl < cw && c0 + cl < len;
        e[u] = ok[u] ? base + (int64_t)l * row_step + c0 + cl : base;
        if constexpr (BF16)
          xv[u] = __uint_as_float((uint32_t)static_cast<const uint16_t*>(grad)[e[u]] << 16);
        else
          xv[u] = static_cast<const float*>(grad)[e[u]];
        hv[u] = h[e[u]];
        gv[u] = g[e[u]];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int l = pass * kGenRowsPerPass + u * 2 + half;
        const float hn = fmaf(eta, xv[u], a * hv[u]);
        if (ok[u]) h[e[u]] = hn;
        tile[l * kGenPitch + cl] = hn - gv[u];
      }
    }
    wave_lds_fence();
    {
      // This row's columns in the chunk: fewer in a ragged last row.  The
      // column loop runs to the chunk width for every lane (V's reads are
      // wave-uniform LDS broadcasts); the lane keeps only its first jn
      // products.  Lanes at or past the row count compute unused values.
      const int64_t len = lane == rows - 1 ? grp.last_len : n;
      const int jn = (int)(len - c0 < cw ? (len - c0 > 0 ? len - c0 : 0) : cw);
      const float* row = tile + lane * kGenPitch;
      float dl[kGenChunk];
#pragma unroll
      for (int j = 0; j < kGenChunk; ++j) dl[j] = row[j];
      for (int32_t k = 0; k < r; ++k) {
        float s = acc[k * kWave + lane];
        const float* vk = vl + k * kGenChunk;
#pragma unroll
        for (int j = 0; j < kGenChunk; ++j) {
          const float t = fmaf(dl[j], norm ? dl[j] : vk[j], s);
          s = j < jn ? t : s;
        }
        acc[k * kWave + lane] = s;
      }
    }
    wave_lds_fence();
  }
  if (lane < rows) {
    float* out = S + ((int64_t)i * m + grp.row0 + (int64_t)lane * grp.stride) * r;
    for (int32_t k = 0; k < r; ++k) out[k] = acc[k * kWave + lane];
  }
}

}  // namespace

hipError_t launch_sketch_general(const void* grad, int32_t grad_bf16, float* h,
                                 const float* g, const float* V, const RowGroup* groups,
                                 int64_t ngroups, float* S, int64_t d, int64_t m, int32_t N,
                                 int32_t r, float eta, float a, bool norm, hipStream_t stream) {
  if (ngroups <= 0) return hipSuccess;
  if (r < 1 || r > ARC_MAX_R) return hipErrorInvalidValue;
  const dim3 grid((unsigned)ngroups, (unsigned)N), block(kWave);
  const size_t lds = sizeof(float) * (kWave + kGenChunk) * r;
  if (grad_bf16)
    hipLaunchKernelGGL(sketch_general_kernel<true>, grid, block, lds, stream, grad, h, g, V,
                       groups, S, d, m, r, eta, a, norm ? 1 : 0);
  else
    hipLaunchKernelGGL(sketch_general_kernel<false>, grid, block, lds, stream, grad, h, g, V,
                       groups, S, d, m, r, eta, a, norm ? 1 : 0);
  return hipGetLastError();
}

}  // namespace arc

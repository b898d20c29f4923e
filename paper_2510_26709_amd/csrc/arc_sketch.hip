// Streaming stage of the compressor step: EF21M momentum (11a), residual
// Delta = h_t - g_{t-1}, per-worker sketch P^(i) = G^(i) V (Alg. 1), worker
// sum and row importance Sigma = diag(P P^T) (Eq. (4)).
//
// Numerics follow the contract in libarctopk.h: binary32; the dot product of
// a row with column k of V is a fused multiply-add chain in ascending column
// order from +0; the worker sum is a chain of plain additions in ascending
// worker order; Sigma is a fused multiply-add chain of squares in ascending k.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "arc_device.h"
#include "arc_internal.h"

namespace arc {
namespace {

// Tile of one wave: 64 rows x 32 columns of Delta, 8 float4 per row plus one
// float4 of padding, so that 16 consecutive lanes reading 16 consecutive rows
// hit 16 distinct 16-byte bank groups; every address is a per-lane base plus
// an immediate offset.
constexpr int kChunk = 32;
constexpr int kRowF4 = 9;
constexpr int kTileF4 = kWave * kRowF4;
__device__ __forceinline__ int tile_slot(int rho, int q) { return rho * kRowF4 + q; }

// One wave's pass over its 64 rows of worker i: loads the grad/h/g tile of
// each 32-column chunk with coalesced 16-byte accesses, applies (11a), writes
// h back, parks Delta in LDS, then runs this lane's r chains over its row.
// FULL: all 64 rows exist (no per-row predicates).
template <int R, bool BF16, bool FULL>
__device__ __forceinline__ void sketch_rows_impl(
    const void* __restrict__ grad, float* __restrict__ h,
    const float* __restrict__ g, const float* __restrict__ V, int64_t d,
    int64_t n, int64_t p0, int64_t row_hi, int32_t i, float eta, float a,
    float4* tile, float (&s)[R]) {
  const int lane = threadIdx.x & (kWave - 1);
  const int sub = lane >> 3;   // row within an 8-row slab
  const int quad = lane & 7;   // 16-byte column group within the chunk
  const int64_t wbase = (int64_t)i * d;
#pragma unroll
  for (int k = 0; k < R; ++k) s[k] = 0.0f;

  const int64_t nchunks = n / kChunk;
  for (int64_t c = 0; c < nchunks; ++c) {
    const int64_t col = c * kChunk + quad * 4;
    float4 xv[8], hv[8], gv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int64_t p = p0 + u * 8 + sub;
      const int64_t e = wbase + p * n + col;
      if (FULL || p < row_hi) {
        if constexpr (BF16) {
          // 8-byte loads cover half a cache line whose other half belongs to
          // the next chunk, so these stay cacheable.  (Counters show about
          // half of those lines leave L2 twice; the second request is served
          // by the last-level cache.  Loading both halves together removes it
          // but costs occupancy and runs no faster.)
          const uint2 w = *reinterpret_cast<const uint2*>(
              static_cast<const uint16_t*>(grad) + e);
          xv[u] = make_float4(bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y));
        } else {
          xv[u] = stream_load(reinterpret_cast<const float4*>(
              static_cast<const float*>(grad) + e));
        }
        hv[u] = *reinterpret_cast<const float4*>(h + e);
        gv[u] = stream_load(reinterpret_cast<const float4*>(g + e));
      } else {
        xv[u] = hv[u] = gv[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      float4 hn;
      hn.x = fmaf(eta, xv[u].x, a * hv[u].x);
      hn.y = fmaf(eta, xv[u].y, a * hv[u].y);
      hn.z = fmaf(eta, xv[u].z, a * hv[u].z);
      hn.w = fmaf(eta, xv[u].w, a * hv[u].w);
      const int64_t p = p0 + u * 8 + sub;
      if (FULL || p < row_hi) stream_store(reinterpret_cast<float4*>(h + wbase + p * n + col), hn);
      float4 dl;
      dl.x = hn.x - gv[u].x;
      dl.y = hn.y - gv[u].y;
      dl.z = hn.z - gv[u].z;
      dl.w = hn.w - gv[u].w;
      tile[tile_slot(u * 8 + sub, quad)] = dl;
    }
    wave_lds_fence();
    const float* Vc = V + c * kChunk * R;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const float4 dv = tile[tile_slot(lane, q)];
      const float e4[4] = {dv.x, dv.y, dv.z, dv.w};
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
#pragma unroll
        for (int k = 0; k < R; ++k)
          s[k] = fmaf(e4[jj], Vc[(q * 4 + jj) * R + k], s[k]);
      }
    }
    wave_lds_fence();
  }
}

template <int R, bool BF16>
__device__ __forceinline__ void sketch_rows(
    const void* __restrict__ grad, float* __restrict__ h,
    const float* __restrict__ g, const float* __restrict__ V, int64_t d,
    int64_t n, int64_t p0, int64_t row_hi, int32_t i, float eta, float a,
    float4* tile, float (&s)[R]) {
  if (p0 + kWave <= row_hi)
    sketch_rows_impl<R, BF16, true>(grad, h, g, V, d, n, p0, row_hi, i, eta, a, tile, s);
  else
    sketch_rows_impl<R, BF16, false>(grad, h, g, V, d, n, p0, row_hi, i, eta, a, tile, s);
}

// ---------------------------------------------------------------------------
// Fused path: a block is N waves, wave i streams worker i over the same 64
// rows; the waves then meet in LDS and wave 0 forms P = S^(0) + S^(1) + ...
// (ascending worker order) and Sigma for its 64 rows.  Sketches never leave
// the chip except as the per-worker copy S kept for inspection.
// HBM traffic per element and worker: grad (4 or 2 B) + h read and write
// (8 B) + g read (4 B).
// ---------------------------------------------------------------------------
template <int R, bool BF16>
__global__ void __launch_bounds__(kMaxFusedWorkers * kWave)
sketch_fused_kernel(const void* __restrict__ grad, float* __restrict__ h,
                    const float* __restrict__ g, const float* __restrict__ V,
                    float* __restrict__ S, float* __restrict__ sigma, int64_t d,
                    int64_t n, int64_t m, int64_t row_lo, int64_t row_hi,
                    int32_t N, float eta, float a) {
  extern __shared__ float4 lds_tiles[];  // N tiles of kTileF4
  const int lane = threadIdx.x & (kWave - 1);
  const int i = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);  // worker
  const int64_t p0 = row_lo + xcd_contiguous_block(blockIdx.x, gridDim.x) * kWave;
  float4* tile = lds_tiles + i * kTileF4;
  float s[R];
  sketch_rows<R, BF16>(grad, h, g, V, d, n, p0, row_hi, i, eta, a, tile, s);
  const int64_t p = p0 + lane;
  if (p < row_hi) {
    float* out = S + ((int64_t)i * m + p) * R;
#pragma unroll
    for (int k = 0; k < R; ++k) out[k] = s[k];
  }
  __syncthreads();  // every wave is done with its tile
  float* comb = reinterpret_cast<float*>(tile);
#pragma unroll
  for (int k = 0; k < R; ++k) comb[k * kWave + lane] = s[k];
  __syncthreads();
  if (i == 0 && p < row_hi) {
    const float* base = reinterpret_cast<const float*>(lds_tiles);
    float acc = 0.0f;
#pragma unroll
    for (int k = 0; k < R; ++k) {
      float P = s[k];
      for (int32_t w = 1; w < N; ++w) P = P + base[w * kTileF4 * 4 + k * kWave + lane];
      acc = fmaf(P, P, acc);
    }
    sigma[p] = acc;
  }
}

// ---------------------------------------------------------------------------
// Per-worker path (more workers than one block holds): same streaming, one
// wave per (64 rows, worker), sketch written to S for the reduce kernel.
// ---------------------------------------------------------------------------
constexpr int kSketchWaves = 4;

template <int R, bool BF16>
__global__ void __launch_bounds__(kSketchWaves * kWave)
sketch_per_worker_kernel(const void* __restrict__ grad, float* __restrict__ h,
                         const float* __restrict__ g, const float* __restrict__ V,
                         float* __restrict__ S, int64_t d, int64_t n, int64_t m,
                         int64_t row_lo, int64_t row_hi, float eta, float a) {
  __shared__ float4 tiles[kSketchWaves][kTileF4];
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int32_t i = blockIdx.y;
  const int64_t p0 =
      row_lo + (xcd_contiguous_block(blockIdx.x, gridDim.x) * kSketchWaves + wave) * kWave;
  if (p0 >= row_hi) return;  // whole wave; no block barrier follows
  float s[R];
  sketch_rows<R, BF16>(grad, h, g, V, d, n, p0, row_hi, i, eta, a, tiles[wave], s);
  const int64_t p = p0 + lane;
  if (p < row_hi) {
    float* out = S + ((int64_t)i * m + p) * R;
#pragma unroll
    for (int k = 0; k < R; ++k) out[k] = s[k];
  }
}

// ---------------------------------------------------------------------------
// General path: one thread per (row, worker); any n, d, r and alignment.  The
// first pass updates h over the row; then, for each k, one pass re-reads h
// (new) and g and runs that column's chain.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256)
sketch_generic_kernel(const void* __restrict__ grad, int32_t grad_bf16,
                      float* __restrict__ h, const float* __restrict__ g,
                      const float* __restrict__ V, float* __restrict__ S,
                      int64_t d, int64_t n, int64_t m, int32_t N, int32_t r,
                      int64_t row_lo, int64_t row_hi, float eta, float a) {
  const int64_t rows = row_hi - row_lo;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= rows * N) return;
  const int32_t i = (int32_t)(tid / rows);
  const int64_t p = row_lo + tid % rows;
  const int64_t base = (int64_t)i * d;
  const int64_t e0 = p * n;
  const int64_t len = (e0 + n <= d) ? n : d - e0;
  for (int64_t j = 0; j < len; ++j) {
    const int64_t e = base + e0 + j;
    float x;
    if (grad_bf16)
      x = __uint_as_float((uint32_t)static_cast<const uint16_t*>(grad)[e] << 16);
    else
      x = static_cast<const float*>(grad)[e];
    h[e] = fmaf(eta, x, a * h[e]);
  }
  for (int32_t k = 0; k < r; ++k) {
    float s = 0.0f;
    for (int64_t j = 0; j < len; ++j) {
      const int64_t e = base + e0 + j;
      const float dl = h[e] - g[e];
      s = fmaf(dl, V[j * r + k], s);
    }
    S[((int64_t)i * m + p) * r + k] = s;
  }
}

// Worker sum and importance from S for rows [row_lo, row_hi); thread per row.
__global__ void __launch_bounds__(256)
reduce_importance_kernel(const float* __restrict__ S, float* __restrict__ sigma,
                         int64_t m, int32_t N, int32_t r, int64_t row_lo,
                         int64_t row_hi) {
  const int64_t p = row_lo + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= row_hi) return;
  float acc = 0.0f;
  if (r == 4) {
    float4 P = *reinterpret_cast<const float4*>(S + p * 4);
    for (int32_t i = 1; i < N; ++i) {
      const float4 q = *reinterpret_cast<const float4*>(S + ((int64_t)i * m + p) * 4);
      P.x = P.x + q.x;
      P.y = P.y + q.y;
      P.z = P.z + q.z;
      P.w = P.w + q.w;
    }
    acc = fmaf(P.x, P.x, acc);
    acc = fmaf(P.y, P.y, acc);
    acc = fmaf(P.z, P.z, acc);
    acc = fmaf(P.w, P.w, acc);
  } else {
    for (int32_t k = 0; k < r; ++k) {
      float P = S[p * r + k];
      for (int32_t i = 1; i < N; ++i) P = P + S[((int64_t)i * m + p) * r + k];
      acc = fmaf(P, P, acc);
    }
  }
  sigma[p] = acc;
}

}  // namespace

size_t fused_sketch_lds_bytes(int32_t N) {
  return (size_t)N * kTileF4 * sizeof(float4);
}

hipError_t launch_sketch_fused(const void* grad, int32_t grad_bf16, float* h,
                               const float* g, const float* V, float* S,
                               float* sigma, int64_t d, int64_t n, int64_t m,
                               int32_t N, int32_t r, int64_t row_lo,
                               int64_t row_hi, float eta, float a,
                               hipStream_t stream) {
  const int64_t rows = row_hi - row_lo;
  if (rows <= 0) return hipSuccess;
  if (N < 1 || N > kMaxFusedWorkers) return hipErrorInvalidValue;
  const dim3 grid(blocks_for(rows, kWave)), block(N * kWave);
  const size_t lds = fused_sketch_lds_bytes(N);
#define ARC_FUSED_CASE(RR)                                                          \
  case RR:                                                                          \
    if (grad_bf16)                                                                  \
      hipLaunchKernelGGL((sketch_fused_kernel<RR, true>), grid, block, lds, stream,  \
                         grad, h, g, V, S, sigma, d, n, m, row_lo, row_hi, N, eta, a); \
    else                                                                            \
      hipLaunchKernelGGL((sketch_fused_kernel<RR, false>), grid, block, lds, stream, \
                         grad, h, g, V, S, sigma, d, n, m, row_lo, row_hi, N, eta, a); \
    break;
  switch (r) {
    ARC_FUSED_CASE(1)
    ARC_FUSED_CASE(2)
    ARC_FUSED_CASE(4)
    ARC_FUSED_CASE(8)
    default:
      return hipErrorInvalidValue;
  }
#undef ARC_FUSED_CASE
  return hipGetLastError();
}

hipError_t launch_sketch(bool fast, const void* grad, int32_t grad_bf16,
                         float* h, const float* g, const float* V, float* S,
                         int64_t d, int64_t n, int64_t m, int32_t N, int32_t r,
                         int64_t row_lo, int64_t row_hi, float eta, float a,
                         hipStream_t stream) {
  const int64_t rows = row_hi - row_lo;
  if (rows <= 0) return hipSuccess;
  if (fast) {
    const dim3 grid(blocks_for(rows, kSketchWaves * kWave), (unsigned)N);
    const dim3 block(kSketchWaves * kWave);
#define ARC_SKETCH_CASE(RR)                                                          \
  case RR:                                                                           \
    if (grad_bf16)                                                                   \
      hipLaunchKernelGGL((sketch_per_worker_kernel<RR, true>), grid, block, 0, stream, \
                         grad, h, g, V, S, d, n, m, row_lo, row_hi, eta, a);         \
    else                                                                             \
      hipLaunchKernelGGL((sketch_per_worker_kernel<RR, false>), grid, block, 0,       \
                         stream, grad, h, g, V, S, d, n, m, row_lo, row_hi, eta, a); \
    break;
    switch (r) {
      ARC_SKETCH_CASE(1)
      ARC_SKETCH_CASE(2)
      ARC_SKETCH_CASE(4)
      ARC_SKETCH_CASE(8)
      default:
        return hipErrorInvalidValue;
    }
#undef ARC_SKETCH_CASE
  } else {
    hipLaunchKernelGGL(sketch_generic_kernel, dim3(blocks_for(rows * N, 256)),
                       dim3(256), 0, stream, grad, grad_bf16, h, g, V, S, d, n,
                       m, N, r, row_lo, row_hi, eta, a);
  }
  return hipGetLastError();
}

hipError_t launch_reduce_importance(const float* S, float* sigma, int64_t m,
                                    int32_t N, int32_t r, int64_t row_lo,
                                    int64_t row_hi, hipStream_t stream) {
  const int64_t rows = row_hi - row_lo;
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(reduce_importance_kernel, dim3(blocks_for(rows, 256)),
                     dim3(256), 0, stream, S, sigma, m, N, r, row_lo, row_hi);
  return hipGetLastError();
}

}  // namespace arc
